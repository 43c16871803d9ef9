"""GPU parity with asymmetric uint8 weights (the ..._plan_create_wt calls,
which legalise them at creation: w - 128 as int8, zero point - 128, as Sec.
III-C legalises a dtype the instructions do not take): conv through every
kernel family, depthwise and dense, against the oracle computing with the
uint8 weights as given."""
import numpy as np
import pytest

import workloads as W
from gpu_util import assert_equal, env, log, make_plan, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

CONV = [
    (W.ConvLayer("u3x3", 13, 11, 64, 96, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    (W.ConvLayer("u3x3s2", 16, 15, 128, 72, 3, 3, 2, (0, 0, 1, 1)), 2, dict(zp_w="tensor", x_dtype="i8")),
    (W.ConvLayer("u1x1", 9, 9, 256, 130, 1, 1), 3, dict(yt="i8")),
    (W.ConvLayer("u_stem", 30, 30, 3, 64, 7, 7, 2, (3, 3, 3, 3)), 2, {}),
    (W.ConvLayer("u_c20", 9, 9, 20, 36, 3, 3, 1, (1, 1, 1, 1)), 2, dict(yt="i32")),
]
FORCED = [{}, dict(QNN_TILE=0), dict(QNN_TAP=0), dict(QNN_DMA=4), dict(QNN_WAVE=2)]


@pytest.mark.parametrize("forced", FORCED, ids=["auto", "gather", "tap", "dma", "wave"])
def test_uint8_weight_conv(forced):
    for i, (layer, N, kw) in enumerate(CONV):
        c = W.conv_case(layer, N, seed=700 + i, w_dtype="u8", **kw)
        assert c.w.dtype == np.uint8 and c.zp_w.min() >= 96
        with env(**forced):
            p, keep = make_plan(c)
            d = p.describe()
            p.close()
            log(f"uint8 w {layer.name} {forced}: {d}")
            assert_equal(run_gpu(c), run_oracle(c), f"{layer.name} {forced}")


def test_uint8_weight_depthwise():
    for i, layer in enumerate([W.ConvLayer("udw", 14, 14, 96, 96, 3, 3, 1, (1, 1, 1, 1), depthwise=True),
                               W.ConvLayer("udw2", 15, 17, 40, 40, 3, 3, 2, (0, 0, 1, 1), depthwise=True),
                               W.ConvLayer("udw5", 9, 9, 12, 12, 5, 5, 1, (2, 2, 2, 2), depthwise=True)]):
        c = W.conv_case(layer, 2, seed=800 + i, w_dtype="u8")
        log(f"uint8 w depthwise {layer.name}")
        assert_equal(run_gpu(c), run_oracle(c), layer.name)


def test_uint8_weight_dense():
    layer = W.ConvLayer("ud", 1, 96, 768, 300, 1, 1)   # 96 tokens x 768 -> 300 as a 1x1 conv
    c = W.conv_case(layer, 1, seed=900, w_dtype="u8", yt="i8")
    dc = W.ConvCase(c.name, c.x.reshape(96, 768), c.s_x, c.zp_x, c.w.reshape(300, 768), c.s_w, c.zp_w, c.bias,
                    c.s_y, c.zp_y, c.yt, c.act, c.rounding, dense=True)
    assert_equal(run_gpu(dc), run_oracle(dc), "dense uint8 w")
