"""Pins of the oracle's requantize (Eq. (5) with the fixed-point multiplier of
Sec. III-B) and qnn.add against exact rational arithmetic, hand-derived
fixtures (tests/golden/requantize_cases.txt) and invariants."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import exact_ref as X
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows():
    rows = []
    with open(os.path.join(GOLDEN, "requantize_cases.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if line:
                rows.append(line)
    return rows


def test_golden_requantize_cases(oracle):
    rows = _golden_rows()
    assert len(rows) >= 20
    for v, M, zp, dt, up, away in rows:
        for mode, expect in (("half_up", up), ("half_away", away)):
            got = oracle.requantize_value(int(v), float(M), int(zp), dt, None, mode)
            assert got == int(expect), (v, M, zp, dt, mode)


def _multipliers(rng, n):
    """Real multipliers over many binades, incl. powers of two, values just
    below a power of two (mantissa rounding up to 2^31) and scale ratios."""
    Ms = [1.0, 0.5, 0.25, 2.0**-20, 2.0**-40, 2.0**-70, 0.75, 1.5, 1000.0, 2.0**29,
          math.nextafter(1.0, 0.0), math.nextafter(0.5, 0.0), 1.0 - 2.0**-33, 0.999999999]
    for _ in range(n):
        s_in = float(np.float32(10.0 ** rng.uniform(-6, 0))) * float(np.float32(10.0 ** rng.uniform(-4, -1)))
        s_out = float(np.float32(10.0 ** rng.uniform(-4, 1)))
        Ms.append(s_in / s_out)
    return Ms


def test_multiplier_representation_bounds(oracle):
    """mult in [2^30, 2^31), shift >= 1 and
    |mult * 2^-shift - M| <= 2^(e-32) for M = f * 2^e (round to nearest of a
    31-bit significand)."""
    rng = np.random.default_rng(1)
    for M in _multipliers(rng, 3000):
        mult, shift = oracle.quantize_multiplier(M)
        assert 2**30 <= mult < 2**31 and shift >= 1
        f, e = math.frexp(M)
        err = abs(Fraction(mult, 2**shift) - Fraction(M))
        assert err <= Fraction(2) ** (e - 32), M


def test_multiplier_rejects_out_of_range(oracle):
    for M in (2.0**30, 2.0**31, float("inf"), float("nan"), -1.0, 2.0**30 - 0.01):
        with pytest.raises(ValueError):
            oracle.quantize_multiplier(M)
    assert oracle.quantize_multiplier(0.0) == (0, 1)


def _check_against_fraction(oracle, M, values, mode):
    mult, shift = oracle.quantize_multiplier(M)
    rnd = X.ROUND[mode]
    for v in values:
        got = oracle.round_mul_shift(v, mult, shift, mode)
        assert got == rnd(Fraction(v * mult, 2**shift)), (M, v, mode)


@pytest.mark.parametrize("mode", ["half_up", "half_away"])
def test_round_mul_shift_exact_rational(oracle, mode):
    """t == round(v * mult / 2^shift) in exact rationals for a dense range of
    v, int32 extremes and constructed ties."""
    rng = np.random.default_rng(2)
    dense = list(range(-4096, 4097))
    extremes = [2**31 - 1, -(2**31), -(2**31) + 1, 2**30, -(2**30), 2**31]
    for M in [0.5, 2.0**-11, 0.75, 0.002, 1.0 / 3.0] + _multipliers(rng, 20):
        _check_against_fraction(oracle, M, dense[:: 1 if M < 2.0**-8 else 7] + extremes, mode)
    # constructed ties: M = 2^-k makes v * M a half-integer for odd v * 2^(1-k) multiples
    for k in range(1, 31):
        M = 2.0**-k
        vs = [(2 * j + 1) * 2 ** (k - 1) for j in range(-20, 20)]
        vs = [v for v in vs if abs(v) <= 2**31]
        _check_against_fraction(oracle, M, vs, mode)


@pytest.mark.parametrize("mode", ["half_up", "half_away"])
def test_requantize_vs_exact_real_multiplier(oracle, mode):
    """Against the exact real multiplier M = s_in/s_out (rationals of the
    binary32 scales), a result may differ only where v*M is within
    |v| * |mult*2^-shift - M| of a tie."""
    rng = np.random.default_rng(3)
    rnd = X.ROUND[mode]
    for _ in range(40):
        s_in = np.float32(10.0 ** rng.uniform(-5, -1))
        s_out = np.float32(10.0 ** rng.uniform(-3, 0))
        M_exact = Fraction(float(s_in)) / Fraction(float(s_out))
        if M_exact >= 2**29:
            continue
        mult, shift = oracle.quantize_multiplier(float(s_in) / float(s_out))
        delta = abs(Fraction(mult, 2**shift) - M_exact)
        vs = rng.integers(-(2**31), 2**31, size=400, dtype=np.int64)
        x = vs.astype(np.int32)
        y = oracle.requantize(x, float(s_in), 0, float(s_out), 0, "i32", None, mode)
        for v, got in zip(x.tolist(), y.tolist()):
            ideal = min(2**31 - 1, max(-(2**31), rnd(Fraction(v) * M_exact)))
            if got != ideal:
                assert abs(got - ideal) == 1
                assert X.is_near_tie(Fraction(v) * M_exact, abs(v) * delta), (v, got, ideal)


def test_requantize_monotone_and_saturating(oracle):
    v = np.arange(-70000, 70001, 7, dtype=np.int32)
    for mode in ("half_up", "half_away"):
        for s_in, s_out, zp, yt in [(0.001, 0.05, 3, "u8"), (0.0123, 0.5, -3, "i8"), (0.3, 0.2, 0, "i32")]:
            y = oracle.requantize(v, s_in, 0, s_out, zp, yt, None, mode).astype(np.int64)
            assert (np.diff(y) >= 0).all()
    y = oracle.requantize(np.array([255, 0], np.uint8), 1.0, 0, 0.001, 0, "u8")
    assert y.tolist() == [255, 0]
    y = oracle.requantize(np.array([127, -128], np.int8), 1.0, 0, 0.001, 0, "i8")
    assert y.tolist() == [127, -128]


def test_unit_multiplier_is_saturating_add(oracle):
    """s_x * s_w / s_y = 1 exactly (0.5 * 0.25 / 0.125) gives y = sat(acc + zp_y)."""
    acc = np.arange(-400, 400, dtype=np.int64).reshape(-1, 8)
    y = oracle.requantize_acc(acc, 0.5, [0.25], 0.125, 17, "u8")
    np.testing.assert_array_equal(y, np.clip(acc + 17, 0, 255).astype(np.uint8))
    y = oracle.requantize_acc(acc, 0.5, [0.25], 0.125, -17, "i8")
    np.testing.assert_array_equal(y, np.clip(acc - 17, -128, 127).astype(np.int8))


def test_relu_clamp_order(oracle):
    """A ReLU (real 0.0) clamp before requantize equals the Q-domain clamp
    lo = zp_y after it: requantize is monotone and maps 0 to zp_y."""
    rng = np.random.default_rng(4)
    acc = rng.integers(-300000, 300000, size=(64, 16)).astype(np.int64)
    s_w = (10.0 ** rng.uniform(-3, -2, size=16)).astype(np.float32)
    for mode in ("half_up", "half_away"):
        after = oracle.requantize_acc(acc, 0.02, s_w, 0.07, 9, "u8", (9, 255), mode)
        before = oracle.requantize_acc(np.maximum(acc, 0), 0.02, s_w, 0.07, 9, "u8", None, mode)
        np.testing.assert_array_equal(after, before)


def test_per_channel_equal_scales_equals_per_tensor(oracle):
    rng = np.random.default_rng(5)
    acc = rng.integers(-10**6, 10**6, size=(50, 12)).astype(np.int64)
    a = oracle.requantize_acc(acc, 0.02, [0.004], 0.3, 5, "u8")
    b = oracle.requantize_acc(acc, 0.02, np.full(12, 0.004, np.float32), 0.3, 5, "u8")
    np.testing.assert_array_equal(a, b)


def test_concat_slice_writes_only_its_channels(oracle):
    rng = np.random.default_rng(6)
    acc = rng.integers(-10**5, 10**5, size=(10, 4)).astype(np.int64)
    out = np.full((10, 9), 200, np.uint8)
    oracle.requantize_acc(acc, 0.02, [0.01], 0.5, 3, "u8", None, "half_up", out=out, y_ldc=9, y_coff=3)
    ref = oracle.requantize_acc(acc, 0.02, [0.01], 0.5, 3, "u8")
    np.testing.assert_array_equal(out[:, 3:7], ref)
    assert (out[:, :3] == 200).all() and (out[:, 7:] == 200).all()


def test_standalone_requantize_per_channel(oracle):
    """Per-channel qparams on the innermost axis equal per-tensor calls on
    each channel slice."""
    rng = np.random.default_rng(7)
    x = rng.integers(0, 256, size=(5, 6, 7), dtype=np.uint8)
    s_in = (10.0 ** rng.uniform(-3, -1, size=7)).astype(np.float32)
    zp_in = rng.integers(0, 256, size=7).astype(np.int32)
    s_out = (10.0 ** rng.uniform(-3, -1, size=7)).astype(np.float32)
    zp_out = rng.integers(-128, 128, size=7).astype(np.int32)
    y = oracle.requantize(x, s_in, zp_in, s_out, zp_out, "i8")
    for c in range(7):
        yc = oracle.requantize(np.ascontiguousarray(x[..., c]), s_in[c], zp_in[c], s_out[c], zp_out[c], "i8")
        np.testing.assert_array_equal(y[..., c], yc)


def test_add_exact_and_invariants(oracle):
    rng = np.random.default_rng(8)
    a = rng.integers(0, 256, size=4096, dtype=np.uint8)
    b = rng.integers(0, 256, size=4096, dtype=np.uint8)
    # equal scales with M = 1: y = sat(zp_o + (a - zp_a) + (b - zp_b))
    y = oracle.add(a, 0.5, 100, b, 0.5, 30, 0.5, 7, "u8")
    ref = np.clip(7 + (a.astype(np.int64) - 100) + (b.astype(np.int64) - 30), 0, 255)
    np.testing.assert_array_equal(y, ref.astype(np.uint8))
    # commutative
    y1 = oracle.add(a, 0.013, 100, b, 0.021, 30, 0.04, 7, "u8")
    y2 = oracle.add(b, 0.021, 30, a, 0.013, 100, 0.04, 7, "u8")
    np.testing.assert_array_equal(y1, y2)
    # against the exact real sum: each input term is rounded once, so the
    # result is within 1 step of round(real / s_o) + zp_o (before saturation)
    s_a, s_b, s_o = (Fraction(float(np.float32(v))) for v in (0.013, 0.021, 0.04))
    for i in range(0, 4096, 13):
        real = s_a * (int(a[i]) - 100) + s_b * (int(b[i]) - 30)
        ideal = min(255, max(0, X.round_half_up(real / s_o) + 7))
        assert abs(int(y1[i]) - ideal) <= 1


def test_add_against_fraction_per_term(oracle):
    """Each input is requantized to the output scale on its own (same
    fixed-point rule as requantize), then summed with zp_o."""
    rng = np.random.default_rng(9)
    case = W.add_case(W.AddLayer("t", 5, 5, 8), 1, seed=3)
    y = oracle.add(case.a, case.s_a, case.zp_a, case.b, case.s_b, case.zp_b, case.s_o, case.zp_o, "u8")
    ma, na = oracle.quantize_multiplier(float(case.s_a) / float(case.s_o))
    mb, nb = oracle.quantize_multiplier(float(case.s_b) / float(case.s_o))
    for i in rng.integers(0, case.a.size, size=300):
        ta = X.round_half_up(Fraction((int(case.a.flat[i]) - case.zp_a) * ma, 2**na))
        tb = X.round_half_up(Fraction((int(case.b.flat[i]) - case.zp_b) * mb, 2**nb))
        assert int(y.flat[i]) == min(255, max(0, case.zp_o + ta + tb))


# ---- the two-stage rounding (Jacob et al.'s integer-only requantize) ----

def test_two_stage_worked_example(oracle):
    """v = 9, M = 2^30 / 2^32 = 1/4: one rounding gives round(2.25) = 2; two
    stages give 9 * 2^30 / 2^31 = 4.5 -> 5 (half up), then 5 / 2 = 2.5 -> 3
    (half away).  v = -9: -4.5 -> -4, -4 / 2 = -2.  v = 7: 3.5 -> 4, 4 / 2 = 2
    (equal to one rounding of 1.75)."""
    m, s = 2**30, 32
    assert oracle.round_mul_shift(9, m, s, "two_stage") == 3
    assert oracle.round_mul_shift(9, m, s, "half_up") == 2
    assert oracle.round_mul_shift(-9, m, s, "two_stage") == -2
    assert oracle.round_mul_shift(7, m, s, "two_stage") == 2
    # stage 2 rounds ties away from zero: -6 * 2^30 / 2^31 = -3 exactly,
    # then -3 / 2 = -1.5 -> -2 (one half-up rounding of -1.5 gives -1)
    assert oracle.round_mul_shift(-6, m, s, "two_stage") == -2
    assert oracle.round_mul_shift(-6, m, s, "half_up") == -1       # -1.5 -> -1
    # shift 31: stage 2 divides by 1, one half-up rounding of v * mult / 2^31
    assert oracle.round_mul_shift(3, 2**30, 31, "two_stage") == 2   # 1.5 -> 2
    assert oracle.round_mul_shift(-3, 2**30, 31, "two_stage") == -1  # -1.5 -> -1


def test_two_stage_exact_rational(oracle):
    """Against the two exact-rational roundings for dense small values, int32
    extremes, constructed stage-1 and stage-2 ties and many multipliers
    (shifts below 31 are one half-up rounding)."""
    rng = np.random.default_rng(12)
    dense = list(range(-3000, 3001, 3))
    extremes = [2**31 - 1, -(2**31), -(2**31) + 1, 2**30, -(2**30), 2**31]
    Ms = [0.5, 0.25, 2.0**-11, 0.75, 0.002, 1.0 / 3.0, 1.5, 3.0, 1000.0] + _multipliers(rng, 30)
    for M in Ms:
        mult, shift = oracle.quantize_multiplier(M)
        for v in dense + extremes + rng.integers(-(2**31), 2**31, size=200).tolist():
            got = oracle.round_mul_shift(v, mult, shift, "two_stage")
            assert got == X.round_two_stage(v * mult, shift), (M, v)
    # ties at each stage: mult = 2^30 makes v * mult / 2^31 = v / 2
    for shift in range(31, 45):
        for v in range(-200, 201):
            assert oracle.round_mul_shift(v, 2**30, shift, "two_stage") == X.round_two_stage(v * 2**30, shift)


def test_two_stage_within_one_of_single_rounding(oracle):
    """Two roundings stay within 1 of one rounding of the same product."""
    rng = np.random.default_rng(13)
    for M in _multipliers(rng, 20):
        mult, shift = oracle.quantize_multiplier(M)
        for v in rng.integers(-(2**31), 2**31, size=300).tolist():
            a = oracle.round_mul_shift(v, mult, shift, "two_stage")
            b = oracle.round_mul_shift(v, mult, shift, "half_up")
            assert abs(a - b) <= 1, (M, v)


def test_two_stage_requantize_monotone(oracle):
    v = np.arange(-70000, 70001, 7, dtype=np.int32)
    for s_in, s_out, zp, yt in [(0.001, 0.05, 3, "u8"), (0.0123, 0.5, -3, "i8"), (0.3, 0.2, 0, "i32")]:
        y = oracle.requantize(v, s_in, 0, s_out, zp, yt, None, "two_stage").astype(np.int64)
        assert (np.diff(y) >= 0).all()
