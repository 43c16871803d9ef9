"""The allocation-free plan run (qnn_plan_run_noalloc, workspace in the
library's static device array) against qnn_plan_run with the plan's own
workspace, byte for byte: two calls in a row through the C ABI, the second
on a smaller input, for plans that use the scratch (split reduction
counters and partial sums, window sums of term 3, the padded image of the
row-pair stem); and the error for a plan whose workspace exceeds it."""
import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import Q, assert_equal, dev, env, log, make_plan, run_oracle

pytestmark = pytest.mark.gpu


def _noalloc(p, x, out):
    st = Q.lib().qnn_plan_run_noalloc(p.handle, None, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr()))
    assert Q.STATUS[st] == "QNN_OK", Q.lib().qnn_last_error().decode()
    return out


CASES = [
    # (layer, batches: first call, then a smaller one; forced kernel, case options)
    (W.ConvLayer("split", 14, 14, 256, 200, 3, 3, 1, (1, 1, 1, 1)), (4, 2), dict(QNN_DMA=0, QNN_KSPLIT=3),
     dict(zp_w="channel")),
    (W.ConvLayer("split_i8", 9, 11, 512, 96, 1, 1), (6, 3), dict(QNN_DMA=4, QNN_KSPLIT=4), dict(yt="i8")),
    (W.ConvLayer("stem", 40, 40, 3, 64, 7, 7, 2, (3, 3, 3, 3)), (3, 1), {}, {}),
]


@pytest.mark.parametrize("layer,batches,forced,kw", CASES, ids=[c[0].name for c in CASES])
def test_noalloc_matches_plan_run(layer, batches, forced, kw):
    for N in batches:
        c = W.conv_case(layer, N, seed=31 + N, **kw)
        with env(**forced):
            p, keep = make_plan(c)
        d = p.describe()
        assert p.workspace_size > 0, d
        x = dev(c.x)
        ref = p.run(x)
        got = torch.full_like(ref, 0x33)
        torch.cuda.synchronize()
        _noalloc(p, x, got)
        torch.cuda.synchronize()
        log(f"noalloc {layer.name} N={N}: {d}")
        assert_equal(got.cpu().numpy(), ref.cpu().numpy(), f"{layer.name} N={N} noalloc vs plan_run")
        assert_equal(got.cpu().numpy(), run_oracle(c), f"{layer.name} N={N} noalloc vs oracle")
        p.close()


def test_noalloc_rejects_oversized_workspace():
    """A split plan whose partial sums need more than the static array."""
    layer = W.ConvLayer("big", 28, 28, 256, 512, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 8, seed=5)
    with env(QNN_DMA=4, QNN_KSPLIT=6):
        p, keep = make_plan(c)
    assert p.workspace_size > (63 << 20), (p.workspace_size, p.describe())
    x = dev(c.x)
    out = p.new_output()
    st = Q.lib().qnn_plan_run_noalloc(p.handle, None, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(out.data_ptr()))
    assert Q.STATUS[st] == "QNN_ERR_UNSUPPORTED"
    assert "static scratch" in Q.lib().qnn_last_error().decode()
    p.close()
