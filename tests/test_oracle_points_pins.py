"""Pins of the oracle's point samplers, the checkers of every large-batch
GPU parity test, against the full-tensor oracle functions (themselves pinned
against exact rationals, the four-term expansion of Eq. (3) and float64
library convolution in the other pin files) and, for requantize, directly
against exact rational arithmetic of Eq. (5):

* conv2d_acc_points equals the full conv2d accumulator at the same flat
  indices, for regular and depthwise (channel multiplier 1) convolutions,
  strided and asymmetrically padded, with per-tensor and per-channel weight
  zero points and uint8 / int8 inputs;
* requantize_points equals requantize_acc at the same flat indices, for
  per-tensor and per-channel weight scales, all three roundings, ReLU and
  ReLU6 clamps and uint8 / int8 / int32 outputs;
* requantize_points of single accumulators equals the exact rational
  value round(v * mult / 2^shift) + zp_y, clamped.
"""
from fractions import Fraction

import numpy as np
import pytest

import exact_ref as X
import workloads as W

ROUNDINGS = ("half_up", "half_away", "two_stage")


def _conv_inputs(rng, depthwise, x_dtype, zpw_mode):
    N, H, Wd = 2, int(rng.integers(5, 12)), int(rng.integers(5, 12))
    C = int(rng.integers(3, 20))
    K = C if depthwise else int(rng.integers(2, 24))
    R, S = int(rng.integers(1, 4)), int(rng.integers(1, 6))
    stride = (int(rng.integers(1, 3)), int(rng.integers(1, 4)))
    pads = tuple(int(v) for v in rng.integers(0, 3, size=4))   # asymmetric
    if x_dtype == "u8":
        x = rng.integers(0, 256, size=(N, H, Wd, C), dtype=np.uint8)
        zp_x = int(rng.integers(0, 256))
    else:
        x = rng.integers(-128, 128, size=(N, H, Wd, C), dtype=np.int8)
        zp_x = int(rng.integers(-128, 128))
    w = (rng.integers(-127, 128, size=(R, S, C), dtype=np.int8) if depthwise
         else rng.integers(-127, 128, size=(K, R, S, C), dtype=np.int8))
    if zpw_mode == "zero":
        zp_w = np.zeros(1, np.int32)
    elif zpw_mode == "tensor":
        zp_w = np.array([int(rng.integers(-20, 21))], np.int32)
    else:
        zp_w = rng.integers(-20, 21, size=K).astype(np.int32)
    bias = rng.integers(-9999, 10000, size=K).astype(np.int32)
    return x, zp_x, w, zp_w, bias, stride, pads


@pytest.mark.parametrize("depthwise", [False, True])
@pytest.mark.parametrize("x_dtype", ["u8", "i8"])
@pytest.mark.parametrize("zpw_mode", ["zero", "tensor", "channel"])
def test_conv_points_equal_full(oracle, depthwise, x_dtype, zpw_mode):
    rng = np.random.default_rng(hash((depthwise, x_dtype, zpw_mode)) % 2**32)
    for _ in range(3):
        x, zp_x, w, zp_w, bias, stride, pads = _conv_inputs(rng, depthwise, x_dtype, zpw_mode)
        full = oracle.conv2d_acc(x, zp_x, w, zp_w, bias, stride, pads, depthwise=depthwise)
        # every index of the small tensor, then a random sample in random order
        idx = np.arange(full.size, dtype=np.int64)
        pts = oracle.conv2d_acc_points(x, zp_x, w, idx, zp_w, bias, stride, pads, depthwise=depthwise)
        np.testing.assert_array_equal(pts, full.reshape(-1))
        idx = rng.permutation(full.size)[: max(1, full.size // 3)].astype(np.int64)
        pts = oracle.conv2d_acc_points(x, zp_x, w, idx, zp_w, bias, stride, pads, depthwise=depthwise)
        np.testing.assert_array_equal(pts, full.reshape(-1)[idx])


def test_depthwise_points_on_a_mobilenet_layer(oracle):
    """A strided MobileNet-V2 depthwise layer (3x3/2, pads 0, 1, 1 ... as
    generated), sampled against the full tensor."""
    layer = [l for l in W.mobilenet_v2_layers() if getattr(l, "depthwise", False) and l.stride == 2][0]
    c = W.conv_case(layer, 2, seed=11, zp_w="channel")
    full = oracle.conv2d_acc(c.x, c.zp_x, c.w, c.zp_w, c.bias, c.stride, c.pads, depthwise=True)
    idx = W.sample_indices(full.size, 5000, seed=12)
    pts = oracle.conv2d_acc_points(c.x, c.zp_x, c.w, idx, c.zp_w, c.bias, c.stride, c.pads, depthwise=True)
    np.testing.assert_array_equal(pts, full.reshape(-1)[idx])


def _acc_and_scales(rng, K, per_channel):
    acc = rng.integers(-2**31, 2**31, size=(37, K), dtype=np.int64)
    acc[0, :] = np.iinfo(np.int32).max
    acc[1, :] = np.iinfo(np.int32).min
    acc[2:6, :] = rng.integers(-3000, 3000, size=(4, K))
    nk = K if per_channel else 1
    s_w = (10.0 ** rng.uniform(-3, -2, size=nk)).astype(np.float32)
    return acc, s_w


@pytest.mark.parametrize("rounding", ROUNDINGS)
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("yt,act", [("u8", None), ("u8", "relu"), ("u8", "relu6"), ("i8", None), ("i8", "relu6"),
                                    ("i32", None)])
def test_requantize_points_equal_full(oracle, rounding, per_channel, yt, act):
    rng = np.random.default_rng(hash((rounding, per_channel, yt, act)) % 2**32)
    K = 19
    acc, s_w = _acc_and_scales(rng, K, per_channel)
    s_x = 0.02
    s_y = float(np.float32(0.25 if yt == "i32" else 3.7))
    zp_y = 0 if yt == "i32" else (17 if yt == "u8" else -5)
    if yt == "i32":
        s_y = float(np.float32(s_x * 1e-2))   # multipliers near 1 for the int32 output
    clamp = None
    if act == "relu":
        clamp = (zp_y, 2**31 - 1)
    elif act == "relu6":
        clamp = (zp_y, zp_y + int(round(6 / s_y)))
    full = oracle.requantize_acc(acc, s_x, s_w, s_y, zp_y, yt, clamp, rounding)
    idx = rng.permutation(acc.size).astype(np.int64)
    pts = oracle.requantize_points(acc.reshape(-1)[idx], idx, K, s_x, s_w, s_y, zp_y, yt, clamp, rounding)
    np.testing.assert_array_equal(pts, full.reshape(-1)[idx].astype(np.int64))


@pytest.mark.parametrize("rounding", ["half_up", "half_away"])
def test_requantize_points_exact_rational(oracle, rounding):
    """Eq. (5) with the fixed-point multiplier: every point is
    clamp(zp_y + round(v * mult / 2^shift)), computed with Fractions from
    the multiplier the oracle derives for that channel."""
    rng = np.random.default_rng(21)
    K = 7
    s_w = (10.0 ** rng.uniform(-3, -2, size=K)).astype(np.float32)
    s_x, s_y, zp_y = 0.02, float(np.float32(0.9)), 3
    v = rng.integers(-2**31, 2**31, size=400, dtype=np.int64)
    idx = rng.integers(0, 10 * K, size=v.size).astype(np.int64)
    got = oracle.requantize_points(v, idx, K, s_x, s_w, s_y, zp_y, "u8", None, rounding)
    rnd = X.round_half_up if rounding == "half_up" else X.round_half_away
    for vi, ii, g in zip(v.tolist(), idx.tolist(), got.tolist()):
        k = ii % K
        M = float(np.float64(np.float32(s_x)) * np.float64(s_w[k]) / np.float64(np.float32(s_y)))
        mult, shift = oracle.quantize_multiplier(M)
        t = rnd(Fraction(vi * mult, 2 ** shift))
        assert g == min(255, max(0, zp_y + t)), (vi, k)
