"""ResNet-50's conv body chained as in the network (stem, max pool, the 16
bottleneck blocks with int8 hand-off and a qnn.add closing every block,
global average pool) on the GPU against the oracle running the same chain on
its own tensors: every one of the 71 intermediate tensors byte for byte."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import Q, O, log, dev, assert_equal  # noqa: E402


def run_chain_gpu(ch):
    t = {"x0": dev(ch.x0)}
    keep = []
    for st in ch.steps:
        if isinstance(st, W.ChainConv):
            s_x, zp_x = ch.q[st.src]
            L = st.layer
            w, b = dev(st.w), dev(st.bias)
            keep += [w, b]
            p = Q.conv2d_plan(tuple(t[st.src].shape), "i8", s_x, zp_x, w, st.s_w, st.zp_w, b, L.stride, L.pads,
                              1, st.s_y, st.zp_y, "i8", st.act)
            out = p.new_output()
            p.run(t[st.src], out)
            torch.cuda.synchronize()
            p.close()
            t[st.dst] = out
        elif isinstance(st, W.ChainPool):
            t[st.dst] = Q.pool2d(t[st.src], st.mode, st.kernel, st.stride, st.pads)
        else:
            s_a, zp_a = ch.q[st.a]
            s_b, zp_b = ch.q[st.b]
            t[st.dst] = Q.add(t[st.a], s_a, zp_a, t[st.b], s_b, zp_b, st.s_o, st.zp_o, "i8", st.act)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in t.items()}


def run_chain_oracle(ch):
    t = {"x0": ch.x0}
    for st in ch.steps:
        if isinstance(st, W.ChainConv):
            s_x, zp_x = ch.q[st.src]
            L = st.layer
            t[st.dst] = O.conv2d(t[st.src], s_x, zp_x, st.w, st.s_w, st.zp_w, st.bias, st.s_y, st.zp_y, "i8",
                                 st.act, "half_up", stride=(L.stride, L.stride), pads=L.pads)
        elif isinstance(st, W.ChainPool):
            t[st.dst] = O.pool2d(t[st.src], st.mode, st.kernel, st.stride, st.pads)
        else:
            s_a, zp_a = ch.q[st.a]
            s_b, zp_b = ch.q[st.b]
            t[st.dst] = O.add(t[st.a], s_a, zp_a, t[st.b], s_b, zp_b, st.s_o, st.zp_o, "i8", st.act)
    return t


@pytest.mark.parametrize("N", [1, 2])
def test_resnet50_chain(N):
    ch = W.resnet50_chain(N)
    log(f"chain N={N}: {len(ch.steps)} steps")
    gpu = run_chain_gpu(ch)
    ref = run_chain_oracle(ch)
    for st in ch.steps:
        assert_equal(gpu[st.dst], ref[st.dst], f"chain N={N} {st.dst}")
    assert len(ch.steps) == 71 and ch.steps[-1].dst == "gap" and ref["gap"].shape == (N, 1, 1, 2048)
    # the data stays informative through the chain: the last block output
    # and the pooled features are neither constant nor all on the clamp
    assert len(np.unique(ref[ch.steps[-2].dst])) > 50
    assert len(np.unique(ref["gap"])) > 20
