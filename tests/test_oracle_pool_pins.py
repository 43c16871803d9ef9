"""Pins of the oracle's quantized pool2d (Eq. (4): scale and zero point pass
through, the quantized input is pooled) against things other than itself:

  * brute force over exact rationals on tiny inputs (the average as a
    Fraction, rounded to nearest by its definition);
  * torch's float64 avg_pool2d / max_pool2d, a library routine: sums of at
    most a few hundred 8-bit values and one correctly rounded division are
    exact enough in binary64 that rounding the float average reproduces the
    exact rounding (a tie k + 1/2 is representable and comes out exactly; a
    non-tie is at least 1/(2*count) from k + 1/2);
  * closed forms: a constant input pools to itself, HALF_AWAY is odd under
    negation, max pooling ignores the order of a window's cells, and the
    dequantized output is within half a step of the real average (Eq. (4)).
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.oracle as O


def _round_fraction(q: Fraction, rounding: str) -> int:
    if rounding == "half_up":
        return math.floor(q + Fraction(1, 2))
    m = math.floor(abs(q) + Fraction(1, 2))
    return -m if q < 0 else m


def _brute(x, mode, kernel, stride, pads, count_pad, zp, rounding):
    N, H, W, C = x.shape
    R, S = kernel
    pt, pl, pb, pr = pads
    Ho, Wo = (H + pt + pb - R) // stride[0] + 1, (W + pl + pr - S) // stride[1] + 1
    y = np.zeros((N, Ho, Wo, C), dtype=x.dtype)
    for n in range(N):
        for oh in range(Ho):
            for ow in range(Wo):
                for c in range(C):
                    cells, padded = [], 0
                    for r in range(R):
                        for s in range(S):
                            h, w = oh * stride[0] - pt + r, ow * stride[1] - pl + s
                            if 0 <= h < H and 0 <= w < W:
                                cells.append(int(x[n, h, w, c]))
                            else:
                                padded += 1
                    if mode == "max":
                        y[n, oh, ow, c] = max(cells)
                    else:
                        vals = cells + ([zp] * padded if count_pad else [])
                        y[n, oh, ow, c] = _round_fraction(Fraction(sum(vals), len(vals)), rounding)
    return y


CASES = [
    # kernel, stride, pads
    ((2, 2), (2, 2), (0, 0, 0, 0)),
    ((3, 3), (1, 1), (1, 1, 1, 1)),
    ((3, 3), (2, 2), (1, 1, 1, 1)),
    ((3, 2), (2, 1), (2, 0, 1, 1)),
    ((1, 3), (1, 2), (0, 2, 0, 1)),
    ((5, 5), (3, 3), (0, 0, 0, 0)),
]


@pytest.mark.parametrize("dt", ["u8", "i8"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_pool_brute_force(dt, case):
    kernel, stride, pads = CASES[case]
    rng = np.random.default_rng(100 + case)
    lo, hi = O.DTYPE_RANGE[dt]
    x = rng.integers(lo, hi + 1, size=(2, 7, 6, 3)).astype(O.NAME_TO_NP[dt])
    zp = int(rng.integers(lo, hi + 1))
    for mode in ("avg", "max"):
        for count_pad in (False, True):
            for rounding in ("half_up", "half_away"):
                got = O.pool2d(x, mode, kernel, stride, pads, count_pad, zp, rounding)
                want = _brute(x, mode, kernel, stride, pads, count_pad, zp, rounding)
                np.testing.assert_array_equal(got, want, f"{mode} pad={count_pad} {rounding}")


def _round_half_away(a):
    return np.sign(a) * np.floor(np.abs(a) + 0.5)


@pytest.mark.parametrize("dt", ["u8", "i8"])
@pytest.mark.parametrize("kernel,stride,pad", [((3, 3), (1, 1), 1), ((3, 3), (2, 2), 1), ((2, 2), (2, 2), 0),
                                               ((7, 7), (1, 1), 0), ((5, 3), (2, 1), 1)])
def test_pool_against_torch_float64(dt, kernel, stride, pad):
    rng = np.random.default_rng(7)
    lo, hi = O.DTYPE_RANGE[dt]
    x = rng.integers(lo, hi + 1, size=(3, 15, 14, 5)).astype(O.NAME_TO_NP[dt])
    zp = int(rng.integers(lo, hi + 1))
    t = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    pads = (pad, pad, pad, pad)
    for count_pad in (False, True):
        # padded cells hold zp: shift so that torch's zero padding is zp
        a = F.avg_pool2d(t - zp, kernel, stride, pad, count_include_pad=count_pad) + zp
        want = _round_half_away(a.permute(0, 2, 3, 1).numpy())
        got = O.pool2d(x, "avg", kernel, stride, pads, count_pad, zp, "half_away")
        np.testing.assert_array_equal(got.astype(np.float64), want)
        want_up = np.floor(a.permute(0, 2, 3, 1).numpy() + 0.5)
        got_up = O.pool2d(x, "avg", kernel, stride, pads, count_pad, zp, "half_up")
        np.testing.assert_array_equal(got_up.astype(np.float64), want_up)
    m = F.max_pool2d(t, kernel, stride, pad).permute(0, 2, 3, 1).numpy()
    np.testing.assert_array_equal(O.pool2d(x, "max", kernel, stride, pads).astype(np.float64), m)


def test_pool_closed_forms():
    rng = np.random.default_rng(11)
    # a constant input pools to itself, whatever the window and padding
    for v in (0, 1, 200, 255):
        x = np.full((1, 9, 8, 4), v, np.uint8)
        for mode in ("avg", "max"):
            y = O.pool2d(x, mode, (3, 3), (2, 2), (1, 1, 1, 1))
            assert (y == v).all()
        # padded cells counted as zp = v change nothing
        assert (O.pool2d(x, "avg", (3, 3), (1, 1), (1, 1, 1, 1), True, v) == v).all()
    # HALF_AWAY is odd: pooling -x gives -(pooling x)
    x = rng.integers(-127, 128, size=(2, 10, 10, 6)).astype(np.int8)
    for k in ((2, 2), (3, 3), (4, 4)):
        a = O.pool2d(x, "avg", k, (1, 1), rounding="half_away").astype(np.int32)
        b = O.pool2d(-x, "avg", k, (1, 1), rounding="half_away").astype(np.int32)
        np.testing.assert_array_equal(a, -b)
    # ties and near-ties of the two roundings: averages 1/2, -1/2 and -3/4
    t = np.zeros((1, 2, 6, 1), np.int8)
    t[0, :, 0:2, 0] = [[1, 0], [0, 1]]        # sum 2 -> 1/2
    t[0, :, 2:4, 0] = [[-1, 0], [0, -1]]      # sum -2 -> -1/2
    t[0, :, 4:6, 0] = [[-1, -1], [0, -1]]     # sum -3 -> -3/4
    up = O.pool2d(t, "avg", (2, 2), (2, 2), rounding="half_up")[0, 0, :, 0]
    away = O.pool2d(t, "avg", (2, 2), (2, 2), rounding="half_away")[0, 0, :, 0]
    assert up.tolist() == [1, 0, -1] and away.tolist() == [1, -1, -1]
    # max ignores the order of a window's cells
    x = rng.integers(0, 256, size=(1, 6, 6, 2)).astype(np.uint8)
    y = O.pool2d(x, "max", (3, 3), (3, 3))
    xp = x.copy()
    for i in range(2):
        for j in range(2):
            blk = xp[0, 3 * i:3 * i + 3, 3 * j:3 * j + 3, :].reshape(9, 2)
            xp[0, 3 * i:3 * i + 3, 3 * j:3 * j + 3, :] = blk[rng.permutation(9)].reshape(3, 3, 2)
    np.testing.assert_array_equal(O.pool2d(xp, "max", (3, 3), (3, 3)), y)
    assert (y[0, :, :, 0] == x[0, :, :, 0].reshape(2, 3, 2, 3).max(axis=(1, 3))).all()


def test_pool_dequantized_within_half_step():
    # Eq. (4): s*(Q_B - zp) is the average of s*(Q_A - zp) up to the output rounding
    rng = np.random.default_rng(12)
    s, zp = 0.037, 17
    x = rng.integers(0, 256, size=(2, 12, 12, 3)).astype(np.uint8)
    y = O.pool2d(x, "avg", (3, 3), (2, 2), (1, 1, 1, 1), True, zp)
    real = F.avg_pool2d(torch.from_numpy(s * (x.astype(np.float64) - zp)).permute(0, 3, 1, 2), 3, 2, 1,
                        count_include_pad=True).permute(0, 2, 3, 1).numpy()
    assert np.abs(s * (y.astype(np.float64) - zp) - real).max() <= s / 2 + 1e-12


def test_pool_empty_window_rejected():
    x = np.zeros((1, 4, 4, 1), np.uint8)
    with pytest.raises(ValueError):
        O.pool2d(x, "avg", (2, 2), (1, 1), (2, 0, 0, 0))
