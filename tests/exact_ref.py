"""Exact-rational reference for tiny inputs (pins the CPU oracle).

Pure Python with ``fractions.Fraction``; no numpy arithmetic, no shared code
with the oracle or the HIP library.  Each function follows the paper's
definitions directly in the real (dequantized) domain:

* Eq. (1): a quantized value Q with (scale, zp) stands for scale * (Q - zp);
  a binary32 scale is converted to its exact rational value.
* Eq. (2): the real convolution of the dequantized tensors, with real 0.0 in
  the padded taps (the real value that the zero-point padding represents).
* Eq. (3): the four integer terms, computed separately.
* Eq. (5): requantize with an exact rational multiplier and an explicit
  rounding rule.
"""
from fractions import Fraction
import math
import struct


def f32(v) -> Fraction:
    """Exact rational value of v rounded to binary32."""
    return Fraction(struct.unpack("<f", struct.pack("<f", float(v)))[0])


def dequantize(q: int, scale, zp: int) -> Fraction:
    return f32(scale) * (int(q) - int(zp))


def out_hw(H, W, R, S, stride, pads):
    pt, pl, pb, pr = pads
    return (H + pt + pb - R) // stride[0] + 1, (W + pl + pr - S) // stride[1] + 1


def conv2d_real(x, s_x, zp_x, w, s_w, zp_w, bias=None, stride=(1, 1), pads=(0, 0, 0, 0)):
    """Real-valued NHWC conv of dequantized tensors (Eq. (2) left-hand side).

    x: nested lists [N][H][W][C] of ints; w: [K][R][S][C]; s_w, zp_w: lists of
    length K; bias: list of K ints with real value bias*s_x*s_w[k].  Padded taps
    hold real 0.0.  Returns nested lists [N][Ho][Wo][K] of Fractions."""
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    K, R, S = len(w), len(w[0]), len(w[0][0])
    Ho, Wo = out_hw(H, W, R, S, stride, pads)
    pt, pl = pads[0], pads[1]
    out = []
    for n in range(N):
        rows = []
        for oh in range(Ho):
            cols = []
            for ow in range(Wo):
                vals = []
                for k in range(K):
                    total = Fraction(0)
                    for r in range(R):
                        for s in range(S):
                            ih, iw = oh * stride[0] + r - pt, ow * stride[1] + s - pl
                            for c in range(C):
                                if 0 <= ih < H and 0 <= iw < W:
                                    a = dequantize(x[n][ih][iw][c], s_x, zp_x)
                                else:
                                    a = Fraction(0)
                                b = dequantize(w[k][r][s][c], s_w[k], zp_w[k])
                                total += a * b
                    if bias is not None:
                        total += int(bias[k]) * f32(s_x) * f32(s_w[k])
                    vals.append(total)
                cols.append(vals)
            rows.append(cols)
        out.append(rows)
    return out


def four_terms(x, zp_x, w, zp_w, stride=(1, 1), pads=(0, 0, 0, 0)):
    """The four terms of Eq. (3), each computed on its own.

    Term 1 convolves the raw quantized values (padded with zp_x), term 2 is
    zp_x times the weight sum, term 3 is zp_w[k] times the input window sum
    (including the zp_x padding), term 4 is J * zp_x * zp_w[k].  Returns a
    dict of nested lists [N][Ho][Wo][K] of ints."""
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    K, R, S = len(w), len(w[0]), len(w[0][0])
    Ho, Wo = out_hw(H, W, R, S, stride, pads)
    pt, pl = pads[0], pads[1]

    def xpad(n, ih, iw, c):
        return x[n][ih][iw][c] if (0 <= ih < H and 0 <= iw < W) else zp_x

    terms = {t: [[[[0] * K for _ in range(Wo)] for _ in range(Ho)] for _ in range(N)]
             for t in ("t1", "t2", "t3", "t4")}
    for n in range(N):
        for oh in range(Ho):
            for ow in range(Wo):
                for k in range(K):
                    t1 = t2 = t3 = t4 = 0
                    for r in range(R):
                        for s in range(S):
                            ih, iw = oh * stride[0] + r - pt, ow * stride[1] + s - pl
                            for c in range(C):
                                t1 += xpad(n, ih, iw, c) * w[k][r][s][c]
                                t2 += zp_x * w[k][r][s][c]
                                t3 += zp_w[k] * xpad(n, ih, iw, c)
                                t4 += zp_x * zp_w[k]
                    terms["t1"][n][oh][ow][k] = t1
                    terms["t2"][n][oh][ow][k] = t2
                    terms["t3"][n][oh][ow][k] = t3
                    terms["t4"][n][oh][ow][k] = t4
    return terms


def round_half_up(q: Fraction) -> int:
    """Nearest integer, ties toward +infinity."""
    return math.floor(q + Fraction(1, 2))


def round_half_away(q: Fraction) -> int:
    """Nearest integer, ties away from zero."""
    m = math.floor(abs(q) + Fraction(1, 2))
    return -m if q < 0 else m


def round_two_stage(p: int, shift: int) -> int:
    """Jacob et al.'s integer-only requantize of the product p = v * mult for
    a right shift `shift`: for shift >= 31, p / 2^31 rounded half up, then
    that integer / 2^(shift - 31) rounded half away from zero; for shift < 31
    one rounding, half up."""
    if shift < 31:
        return round_half_up(Fraction(p, 2**shift))
    x1 = round_half_up(Fraction(p, 2**31))
    return round_half_away(Fraction(x1, 2**(shift - 31)))


ROUND = {"half_up": round_half_up, "half_away": round_half_away}


def is_near_tie(q: Fraction, tol: Fraction) -> bool:
    """True when q lies within tol of a half-integer."""
    frac = q - math.floor(q)
    return abs(frac - Fraction(1, 2)) <= tol
