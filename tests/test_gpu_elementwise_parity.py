"""GPU parity of standalone requantize and qnn.add against the oracle."""
import zlib

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import Q, O, log, dev, assert_equal  # noqa: E402

_NP = {"u8": np.uint8, "i8": np.int8, "i32": np.int32}
_RANGE = {"u8": (0, 256), "i8": (-128, 128), "i32": (-(2**31), 2**31)}


def _draw(rng, dt, shape):
    lo, hi = _RANGE[dt]
    return rng.integers(lo, hi, size=shape, dtype=np.int64).astype(_NP[dt])


@pytest.mark.parametrize("xt", ["u8", "i8", "i32"])
@pytest.mark.parametrize("yt", ["u8", "i8", "i32"])
@pytest.mark.parametrize("perch", [False, True])
def test_requantize(xt, yt, perch):
    rng = np.random.default_rng(zlib.crc32(f"{xt}{yt}{perch}".encode()))
    for shape in [(3, 5, 7, 33), (1000003,), (2, 16), (64, 96)]:
        x = _draw(rng, xt, shape)
        C = shape[-1]
        n = C if perch else 1
        s_in = (10.0 ** rng.uniform(-3, -1, size=n)).astype(np.float32)
        if xt == "i32":
            s_in = (10.0 ** rng.uniform(-7, -5, size=n)).astype(np.float32)
        zp_in = np.zeros(n, np.int32) if xt == "i32" else _draw(rng, xt, n).astype(np.int32)
        s_out = (10.0 ** rng.uniform(-3, -1, size=n)).astype(np.float32)
        zp_out = np.zeros(n, np.int32) if yt == "i32" else _draw(rng, yt, n).astype(np.int32)
        for rounding in ("half_up", "half_away", "two_stage"):
            log(f"requantize {xt}->{yt} perch={perch} {shape} {rounding}")
            act = None if yt == "i32" else (int(zp_out.min()), _RANGE[yt][1] - 1)
            y = Q.requantize(dev(x), s_in, zp_in, s_out, zp_out, yt, act, rounding).cpu().numpy()
            ref = O.requantize(x, s_in, zp_in, s_out, zp_out, yt, act, rounding)
            assert_equal(y, ref, f"requantize {xt}->{yt} {shape}")


def test_requantize_plan_and_unaligned():
    rng = np.random.default_rng(3)
    x = _draw(rng, "i32", (4, 7, 7, 64))
    s_in = (10.0 ** rng.uniform(-7, -6, size=64)).astype(np.float32)
    zp_in = np.zeros(64, np.int32)
    p = Q.requantize_plan(x.shape, "i32", s_in, zp_in, 0.05, 10, "u8")
    y = p.run(dev(x)).cpu().numpy()
    ref = O.requantize(x, s_in, zp_in, 0.05, 10, "u8")
    assert_equal(y, ref, "requantize plan")
    p.close()
    # unaligned (odd offset) views of uint8 data take the scalar path
    xb = _draw(rng, "u8", 4099)
    xd = dev(xb)
    y = Q.requantize(xd[3:], 0.02, 7, 0.05, 1, "i8").cpu().numpy()
    assert_equal(y, O.requantize(xb[3:], 0.02, 7, 0.05, 1, "i8"), "unaligned")


def test_add_mobilenet_residuals_batch64():
    layers = [l for l in W.mobilenet_v2_layers() if isinstance(l, W.AddLayer)]
    for i, layer in enumerate(layers):
        c = W.add_case(layer, 64, seed=40 + i)
        log(f"add {layer.name}")
        y = Q.add(dev(c.a), c.s_a, c.zp_a, dev(c.b), c.s_b, c.zp_b, c.s_o, c.zp_o, c.yt).cpu().numpy()
        assert_equal(y, O.add(c.a, c.s_a, c.zp_a, c.b, c.s_b, c.zp_b, c.s_o, c.zp_o, c.yt), layer.name)


@pytest.mark.parametrize("at,bt,yt", [("u8", "u8", "u8"), ("i8", "u8", "i8"), ("i8", "i8", "u8")])
def test_add_variants(at, bt, yt):
    rng = np.random.default_rng(4)
    for count in (1, 15, 16, 17, 100003):
        a, b = _draw(rng, at, count), _draw(rng, bt, count)
        za, zb = int(_draw(rng, at, 1)[0]), int(_draw(rng, bt, 1)[0])
        zo = int(_draw(rng, yt, 1)[0])
        for rounding in ("half_up", "half_away", "two_stage"):
            act = (zo, _RANGE[yt][1] - 1)
            y = Q.add(dev(a), 0.013, za, dev(b), 0.3, zb, 0.021, zo, yt, act, rounding).cpu().numpy()
            ref = O.add(a, 0.013, za, b, 0.3, zb, 0.021, zo, yt, act, rounding)
            assert_equal(y, ref, f"add {at}+{bt}->{yt} n={count}")


@pytest.mark.parametrize("yt", ["i8", "i32"])
def test_requantize_two_stage_ties(yt):
    """Scale ratios 1/4, 3/8 and 5/1024 put many products on a tie of the
    first or the second rounding, where the two-stage result differs from
    one half-up rounding; the GPU follows the oracle on every one."""
    rng = np.random.default_rng(21)
    x = rng.integers(-500, 500, size=(4099,), dtype=np.int64).astype(np.int32)   # int8 results mostly unclamped
    differs = 0
    for s_in, s_out in [(0.25, 1.0), (0.375, 1.0), (5.0, 1024.0)]:
        y = Q.requantize(dev(x), s_in, 0, s_out, 0, yt, None, "two_stage").cpu().numpy()
        ref = O.requantize(x, s_in, 0, s_out, 0, yt, None, "two_stage")
        assert_equal(y, ref, f"two-stage ties {s_in}/{s_out}")
        differs += int((ref != O.requantize(x, s_in, 0, s_out, 0, yt, None, "half_up")).sum())
    assert differs > 1000


@pytest.mark.parametrize("ratio", [2.0**13 * 1.5, 2.0**-10 * 1.5, 2.0**14 * 1.5, 2.0**-11 * 1.5, 0.62, 1.0,
                                   2.0**23 * 1.5])
def test_add_shift_range(ratio):
    """Input / output scale ratios whose fixed-point shifts sit at the edges
    of the 24-bit product form of the add (shifts 17 and 40) and just
    outside it (16 and 41: the 64-bit form), for every pair of input bytes;
    the last ratio makes a term exceed 2^30, where the kernel adds without
    its per-byte term tables."""
    a = np.repeat(np.arange(256, dtype=np.int32), 256).astype(np.uint8)
    b = np.tile(np.arange(256, dtype=np.int32), 256).astype(np.uint8)
    s_o = 0.01
    s_a = float(np.float32(ratio * s_o))
    s_b = float(np.float32(0.37 * s_o))
    for rounding in ("half_up", "half_away"):
        y = Q.add(dev(a), s_a, 131, dev(b), s_b, 7, s_o, -5, "i8", None, rounding).cpu().numpy()
        ref = O.add(a, s_a, 131, b, s_b, 7, s_o, -5, "i8", None, rounding)
        assert_equal(y, ref, f"add ratio {ratio} {rounding}")
