"""Quantized pool2d (Eq. (4)) on the GPU against the oracle, byte for byte:
the pooling layers of ResNet-50, MobileNet-V2 and Inception-v3 at their
batch sizes, random shapes over the 16-, 4- and 1-channel paths, asymmetric
padding, both roundings, counted padding, unaligned views, an empty batch,
a window too large for int16 sums, and the rejected arguments."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import Q, O, log, dev, assert_equal  # noqa: E402


def _rand(rng, shape, dt):
    lo, hi = O.DTYPE_RANGE[dt]
    return rng.integers(lo, hi + 1, size=shape).astype(O.NAME_TO_NP[dt])


def _run(x, mode, kernel, stride, pads, count_pad=False, zp=0, rounding="half_away"):
    y = Q.pool2d(dev(x), mode, kernel, stride, pads, count_pad, zp, rounding)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# (name, N, H, W, C, mode, kernel, stride, pads, count_pad)
NETWORK = [
    ("resnet50 stem max 3x3/2", 32, 112, 112, 64, "max", (3, 3), (2, 2), (1, 1, 1, 1), False),
    ("resnet50 global avg 7x7", 32, 7, 7, 2048, "avg", (7, 7), (1, 1), (0, 0, 0, 0), False),
    ("mobilenet_v2 global avg 7x7", 64, 7, 7, 1280, "avg", (7, 7), (1, 1), (0, 0, 0, 0), False),
    ("inception max 3x3/2 147", 64, 147, 147, 64, "max", (3, 3), (2, 2), (0, 0, 0, 0), False),
    ("inception max 3x3/2 71", 64, 71, 71, 192, "max", (3, 3), (2, 2), (0, 0, 0, 0), False),
    ("inception branch avg 3x3 35", 64, 35, 35, 192, "avg", (3, 3), (1, 1), (1, 1, 1, 1), False),
    ("inception branch avg 3x3 17", 64, 17, 17, 768, "avg", (3, 3), (1, 1), (1, 1, 1, 1), False),
    ("inception branch avg 3x3 8 counted", 64, 8, 8, 1280, "avg", (3, 3), (1, 1), (1, 1, 1, 1), True),
    ("inception global avg 8x8", 64, 8, 8, 2048, "avg", (8, 8), (1, 1), (0, 0, 0, 0), False),
]


@pytest.mark.parametrize("dt", ["u8", "i8"])
@pytest.mark.parametrize("case", range(len(NETWORK)))
def test_network_pooling_layers(dt, case):
    name, N, H, W, C, mode, kernel, stride, pads, count_pad = NETWORK[case]
    rng = np.random.default_rng(7000 + case)
    x = _rand(rng, (N, H, W, C), dt)
    zp = int(rng.integers(*O.DTYPE_RANGE[dt]))
    log(f"pool {name} {dt} N={N}")
    got = _run(x, mode, kernel, stride, pads, count_pad, zp)
    want = O.pool2d(x, mode, kernel, stride, pads, count_pad, zp)
    assert_equal(got, want, f"{name} {dt}")


@pytest.mark.parametrize("C", [32, 48, 12, 20, 7, 1, 33])
def test_random_shapes(C):
    rng = np.random.default_rng(7100 + C)
    for it in range(6):
        dt = ["u8", "i8"][it % 2]
        N, H, W = int(rng.integers(1, 4)), int(rng.integers(1, 24)), int(rng.integers(1, 24))
        R, S = int(rng.integers(1, min(H, 5) + 1)), int(rng.integers(1, min(W, 5) + 1))
        pads = tuple(int(rng.integers(0, k)) for k in (R, S, R, S))
        stride = (int(rng.integers(1, 4)), int(rng.integers(1, 4)))
        x = _rand(rng, (N, H, W, C), dt)
        zp = int(rng.integers(*O.DTYPE_RANGE[dt]))
        for mode in ("avg", "max"):
            for count_pad in (False, True):
                for rounding in ("half_up", "half_away"):
                    tag = f"C={C} it={it} {dt} {mode} k={R}x{S} s={stride} p={pads} cp={count_pad} {rounding}"
                    got = _run(x, mode, (R, S), stride, pads, count_pad, zp, rounding)
                    want = O.pool2d(x, mode, (R, S), stride, pads, count_pad, zp, rounding)
                    assert_equal(got, want, tag)


def test_rounding_ties_both_modes():
    # windows of two cells: every odd sum is a tie, of either sign
    rng = np.random.default_rng(7200)
    x = _rand(rng, (2, 9, 16, 64), "i8")
    for rounding in ("half_up", "half_away"):
        got = _run(x, "avg", (1, 2), (1, 2), (0, 0, 0, 0), rounding=rounding)
        want = O.pool2d(x, "avg", (1, 2), (1, 2), (0, 0, 0, 0), rounding=rounding)
        assert_equal(got, want, rounding)
    up = O.pool2d(x, "avg", (1, 2), (1, 2), rounding="half_up")
    away = O.pool2d(x, "avg", (1, 2), (1, 2), rounding="half_away")
    assert (up != away).sum() > 1000


def test_unaligned_views():
    rng = np.random.default_rng(7300)
    for dt in ("u8", "i8"):
        x = _rand(rng, (2 * 10 * 10 * 64 + 1,), dt)
        xd = dev(x)[1:].view(2, 10, 10, 64)
        out = torch.empty(2 * 5 * 5 * 64 + 1, dtype=xd.dtype, device=xd.device)[1:].view(2, 5, 5, 64)
        for mode in ("avg", "max"):
            Q.pool2d(xd, mode, (3, 3), (2, 2), (1, 1, 1, 1), out=out)
            torch.cuda.synchronize()
            want = O.pool2d(x[1:].reshape(2, 10, 10, 64), mode, (3, 3), (2, 2), (1, 1, 1, 1))
            assert_equal(out.cpu().numpy(), want, f"unaligned {dt} {mode}")


def test_large_window_and_empty_batch():
    rng = np.random.default_rng(7400)
    # 17x17 window: sums up to 289*255, beyond int16
    x = np.full((2, 17, 17, 16), 255, np.uint8)
    x[1] = _rand(rng, (17, 17, 16), "u8")
    assert_equal(_run(x, "avg", (17, 17), (1, 1), (0, 0, 0, 0)),
                 O.pool2d(x, "avg", (17, 17), (1, 1), (0, 0, 0, 0)), "17x17 window")
    e = Q.pool2d(torch.empty((0, 8, 8, 16), dtype=torch.uint8, device="cuda"), "avg", (3, 3), (1, 1), 1)
    torch.cuda.synchronize()
    assert tuple(e.shape) == (0, 8, 8, 16)


def test_rejected_arguments():
    x = torch.zeros((1, 8, 8, 16), dtype=torch.uint8, device="cuda")
    with pytest.raises(Q.QnnError):
        Q.pool2d(x, "avg", (3, 3), (1, 1), (3, 0, 0, 0))          # a window with no input cell
    with pytest.raises(Q.QnnError):
        Q.pool2d(x, "avg", (3, 3), (1, 1), 1, rounding="two_stage")
    with pytest.raises(Q.QnnError):
        Q.pool2d(x, "avg", (3, 3), (1, 1), 1, count_pad=True, zp=300)
    with pytest.raises(Q.QnnError):
        Q.pool2d(x, "avg", (9, 3), (1, 1), 0)                     # window larger than the input
    torch.cuda.synchronize()


@pytest.mark.parametrize("dt", ["u8", "i8"])
def test_packed_sum_window_bounds(dt):
    # windows of 257 cells (the largest whose byte sums the kernel packs two
    # to a register: 257 * 255 = 65535) and of 272 cells (summed unpacked),
    # on outputs large enough for the one-pixel-per-thread kernel
    rng = np.random.default_rng(7500)
    hi = O.DTYPE_RANGE[dt][1]
    for (N, H, W, R, S) in ((6, 64, 300, 1, 257), (28, 40, 40, 16, 17)):
        for fill in ("max", "random"):
            if fill == "max":
                x = np.full((N, H, W, 64), hi, O.NAME_TO_NP[dt])
            else:
                x = _rand(rng, (N, H, W, 64), dt)
            for rounding in ("half_up", "half_away"):
                tag = f"{dt} {R}x{S} {fill} {rounding}"
                log(f"pool {tag}")
                got = _run(x, "avg", (R, S), (1, 1), (0, 0, 0, 0), rounding=rounding)
                assert_equal(got, O.pool2d(x, "avg", (R, S), (1, 1), (0, 0, 0, 0), rounding=rounding), tag)
