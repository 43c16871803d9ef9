"""Pins of the oracle's accumulators (conv2d, depthwise, dense) against what
the paper and the mathematics fix, independent of the oracle's own code:

* exact-rational dequantize identity, Eq. (1)/(2): the real convolution of
  the dequantized tensors (real 0.0 in the padding) equals s_x*s_w[k]*acc;
* the four-term expansion, Eq. (3), computed term by term;
* float64 library convolution (all partial sums are integers < 2^53);
* closed forms derived by hand (tests/golden/conv_closed_form.txt);
* special-case reductions (1x1 conv = dense, depthwise = grouped conv,
  full-window conv = dense over the flattened window);
* uint8 -> int8 legalisation invariance (Sec. III-C).
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import exact_ref as X
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_case(rng, x_dtype="u8", per_channel=True, zp_w_nonzero=True, bias=True):
    N = int(rng.integers(1, 3))
    H, Wd = int(rng.integers(2, 6)), int(rng.integers(2, 6))
    C, K = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    R, S = int(rng.integers(1, min(H, 3) + 1)), int(rng.integers(1, min(Wd, 3) + 1))
    stride = (int(rng.integers(1, 3)), int(rng.integers(1, 3)))
    pads = tuple(int(v) for v in rng.integers(0, 3, size=4))
    if x_dtype == "u8":
        x = rng.integers(0, 256, size=(N, H, Wd, C), dtype=np.uint8)
        zp_x = int(rng.integers(0, 256))
    else:
        x = rng.integers(-128, 128, size=(N, H, Wd, C), dtype=np.int8)
        zp_x = int(rng.integers(-128, 128))
    w = rng.integers(-128, 128, size=(K, R, S, C), dtype=np.int8)
    nk = K if per_channel else 1
    s_w = (10.0 ** rng.uniform(-3, -1, size=nk)).astype(np.float32)
    zp_w = rng.integers(-30, 31, size=nk).astype(np.int32) if zp_w_nonzero else np.zeros(nk, np.int32)
    b = rng.integers(-5000, 5001, size=K).astype(np.int32) if bias else None
    s_x = np.float32(10.0 ** rng.uniform(-3, -1))
    return dict(x=x, zp_x=zp_x, s_x=float(s_x), w=w, s_w=s_w, zp_w=zp_w, bias=b,
                stride=stride, pads=pads)


@pytest.mark.parametrize("seed", range(12))
def test_dequantize_identity_exact_rationals(oracle, seed):
    """Eq. (2): C_fp32 = s_A * s_B * Q_C with real 0.0 padding (Eq. (1))."""
    rng = np.random.default_rng(100 + seed)
    c = _tiny_case(rng, x_dtype="u8" if seed % 2 == 0 else "i8", per_channel=seed % 3 != 0,
                   zp_w_nonzero=seed % 4 != 1, bias=seed % 5 != 2)
    acc = oracle.conv2d_acc(c["x"], c["zp_x"], c["w"], c["zp_w"], c["bias"], c["stride"], c["pads"])
    K = c["w"].shape[0]
    s_w = np.broadcast_to(c["s_w"], (K,)).tolist()
    zp_w = np.broadcast_to(c["zp_w"], (K,)).tolist()
    real = X.conv2d_real(c["x"].tolist(), c["s_x"], c["zp_x"], c["w"].tolist(), s_w, zp_w,
                         None if c["bias"] is None else c["bias"].tolist(), c["stride"], c["pads"])
    N, Ho, Wo, _ = acc.shape
    assert (N, Ho, Wo) == (len(real), len(real[0]), len(real[0][0]))
    for n in range(N):
        for oh in range(Ho):
            for ow in range(Wo):
                for k in range(K):
                    lhs = real[n][oh][ow][k]
                    rhs = X.f32(c["s_x"]) * X.f32(s_w[k]) * int(acc[n, oh, ow, k])
                    assert lhs == rhs, (n, oh, ow, k)


@pytest.mark.parametrize("seed", range(8))
def test_four_term_expansion(oracle, seed):
    """Eq. (3): acc = t1 - t2 - t3 + t4 with zp padding, term by term."""
    rng = np.random.default_rng(200 + seed)
    c = _tiny_case(rng, x_dtype="u8" if seed % 2 else "i8", bias=False)
    acc = oracle.conv2d_acc(c["x"], c["zp_x"], c["w"], c["zp_w"], None, c["stride"], c["pads"])
    K = c["w"].shape[0]
    zp_w = np.broadcast_to(c["zp_w"], (K,)).tolist()
    T = X.four_terms(c["x"].tolist(), c["zp_x"], c["w"].tolist(), zp_w, c["stride"], c["pads"])
    combined = (np.array(T["t1"]) - np.array(T["t2"]) - np.array(T["t3"]) + np.array(T["t4"]))
    np.testing.assert_array_equal(combined, acc)
    # terms 2 and 4 depend only on k (compile-time constants, Sec. III-B)
    t2, t4 = np.array(T["t2"]), np.array(T["t4"])
    assert (t2 == t2[:1, :1, :1, :]).all() and (t4 == t4[:1, :1, :1, :]).all()


def _torch_conv_acc(x, zp_x, w, zp_w, stride, pads, dil=(1, 1), groups=1):
    """float64 conv of (x - zp_x) with zero padding and (w - zp_w); exact."""
    xt = torch.from_numpy(x.astype(np.float64) - zp_x).permute(0, 3, 1, 2)
    if groups == 1:
        wt = torch.from_numpy(w.astype(np.float64) - np.asarray(zp_w).reshape(-1, 1, 1, 1)).permute(0, 3, 1, 2)
    else:  # depthwise [R][S][C] -> [C][1][R][S]
        wt = torch.from_numpy(w.astype(np.float64) - np.asarray(zp_w).reshape(1, 1, -1)).permute(2, 0, 1).unsqueeze(1)
    pt, pl, pb, pr = pads
    xt = F.pad(xt, (pl, pr, pt, pb))
    y = F.conv2d(xt, wt, stride=stride, dilation=dil, groups=groups)
    return y.permute(0, 2, 3, 1).numpy()


FULL_LAYERS = [
    W.SINGLE_CONV,
    W.resnet50()[0],                                   # stem 7x7/2, Cin 3
    [l for l in W.resnet50() if l.name == "s28b0_3x3"][0],   # 3x3 stride 2
    [l for l in W.inception_v3() if l.name == "mixed6b_b2_1x7"][0],
    [l for l in W.inception_v3() if l.name == "mixed6b_b2_7x1"][0],
    [l for l in W.mobilenet_v2_layers() if l.name == "c24_0_dw"][0],   # dw s2, asym pads
    [l for l in W.mobilenet_v2_layers() if l.name == "c32_1_dw"][0],   # dw s1
]


@pytest.mark.parametrize("layer", FULL_LAYERS, ids=lambda l: l.name)
def test_float64_library_conv_full_layer(oracle, layer):
    """Full-size layer shapes (batch 1): torch float64 conv is exact here."""
    c = W.conv_case(layer, 1, seed=7, zp_w="channel")
    acc = oracle.conv2d_acc(c.x, c.zp_x, c.w, c.zp_w, c.bias, c.stride, c.pads,
                            depthwise=c.depthwise)
    ref = _torch_conv_acc(c.x, c.zp_x, c.w, c.zp_w, c.stride, c.pads,
                          groups=c.K if c.depthwise else 1)
    ref = ref + (0 if c.bias is None else c.bias.astype(np.float64))
    assert np.abs(ref).max() < 2**53
    np.testing.assert_array_equal(acc, ref.astype(np.int64))


@pytest.mark.parametrize("dil", [(2, 1), (1, 3), (2, 2)])
def test_dilation_matches_library(oracle, dil):
    rng = np.random.default_rng(11)
    x = rng.integers(0, 256, size=(2, 9, 10, 5), dtype=np.uint8)
    w = rng.integers(-127, 128, size=(4, 3, 2, 5), dtype=np.int8)
    zp_w = np.array([1, -2, 0, 5], np.int32)
    acc = oracle.conv2d_acc(x, 17, w, zp_w, None, (1, 2), (1, 0, 2, 1), dil)
    ref = _torch_conv_acc(x, 17, w, zp_w, (1, 2), (1, 0, 2, 1), dil)
    np.testing.assert_array_equal(acc, ref.astype(np.int64))


def test_dense_matches_float64_matmul(oracle):
    c = W.dense_case(W.bert_ffn()[0], seed=2)
    acc = oracle.dense_acc(c.x, c.zp_x, c.w, c.zp_w, None)
    ref = (c.x.astype(np.float64) - c.zp_x) @ (c.w.astype(np.float64) - c.zp_w[:, None]).T
    np.testing.assert_array_equal(acc, ref.astype(np.int64))


def test_golden_closed_form(oracle):
    """Hand-derived values (tests/golden/conv_closed_form.txt)."""
    rows = []
    with open(os.path.join(GOLDEN, "conv_closed_form.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if line:
                rows.append(line)
    assert len(rows) >= 5
    for dt, a, z, b, corner, edge, centre in rows:
        npdt = np.uint8 if dt == "u8" else np.int8
        x = np.full((1, 3, 3, 1), int(a), npdt)
        w = np.full((1, 3, 3, 1), int(b), np.int8)
        acc = oracle.conv2d_acc(x, int(z), w, 0, None, (1, 1), (1, 1, 1, 1))[0, :, :, 0]
        expect = np.array([[corner, edge, corner], [edge, centre, edge], [corner, edge, corner]],
                          dtype=np.int64)
        np.testing.assert_array_equal(acc, expect.astype(np.int64), err_msg=str((dt, a, z, b)))


def test_one_by_one_conv_equals_dense(oracle):
    rng = np.random.default_rng(5)
    x = rng.integers(0, 256, size=(3, 7, 5, 24), dtype=np.uint8)
    w = rng.integers(-127, 128, size=(40, 1, 1, 24), dtype=np.int8)
    zp_w = rng.integers(-9, 10, size=40).astype(np.int32)
    bias = rng.integers(-999, 1000, size=40).astype(np.int32)
    conv = oracle.conv2d_acc(x, 99, w, zp_w, bias)
    dense = oracle.dense_acc(x.reshape(-1, 24), 99, w.reshape(40, 24), zp_w, bias)
    np.testing.assert_array_equal(conv.reshape(-1, 40), dense)


def test_full_window_conv_equals_dense(oracle):
    rng = np.random.default_rng(6)
    x = rng.integers(-128, 128, size=(4, 3, 5, 6), dtype=np.int8)
    w = rng.integers(-127, 128, size=(7, 3, 5, 6), dtype=np.int8)
    conv = oracle.conv2d_acc(x, -5, w, 3, None)
    dense = oracle.dense_acc(x.reshape(4, -1), -5, w.reshape(7, -1), 3, None)
    np.testing.assert_array_equal(conv.reshape(4, 7), dense)


def test_depthwise_equals_block_diagonal_conv(oracle):
    """Depthwise (channel multiplier 1) is the conv whose output channel k
    uses only input channel k."""
    rng = np.random.default_rng(8)
    C = 6
    x = rng.integers(0, 256, size=(2, 6, 7, C), dtype=np.uint8)
    wd = rng.integers(-127, 128, size=(3, 3, C), dtype=np.int8)
    zp_w = rng.integers(-5, 6, size=C).astype(np.int32)
    bias = rng.integers(-99, 100, size=C).astype(np.int32)
    # block-diagonal dense weights with the zero point placed off the diagonal
    # so that (w - zp_w) vanishes there
    wfull = np.empty((C, 3, 3, C), np.int8)
    for k in range(C):
        wfull[k] = zp_w[k]
        wfull[k, :, :, k] = wd[:, :, k]
    for stride, pads in [((1, 1), (1, 1, 1, 1)), ((2, 2), (0, 0, 1, 1)), ((2, 1), (1, 2, 0, 1))]:
        dw = oracle.conv2d_acc(x, 77, wd, zp_w, bias, stride, pads, depthwise=True)
        full = oracle.conv2d_acc(x, 77, wfull, zp_w, bias, stride, pads)
        np.testing.assert_array_equal(dw, full)


@pytest.mark.parametrize("depthwise", [False, True])
def test_legalisation_invariance(oracle, depthwise):
    """Sec. III-C legalisation: uint8 (Q, zp) and int8 (Q-128, zp-128) give
    identical accumulators."""
    rng = np.random.default_rng(9)
    x = rng.integers(0, 256, size=(2, 8, 8, 16), dtype=np.uint8)
    w = (rng.integers(-127, 128, size=(3, 3, 16), dtype=np.int8) if depthwise
         else rng.integers(-127, 128, size=(12, 3, 3, 16), dtype=np.int8))
    xi = (x.astype(np.int16) - 128).astype(np.int8)
    a = oracle.conv2d_acc(x, 200, w, 2, None, (1, 1), (1, 1, 1, 1), depthwise=depthwise)
    b = oracle.conv2d_acc(xi, 72, w, 2, None, (1, 1), (1, 1, 1, 1), depthwise=depthwise)
    np.testing.assert_array_equal(a, b)


def test_points_match_full(oracle):
    layer = [l for l in W.inception_v3() if l.name == "mixed5b_b2_5x5"][0]
    c = W.conv_case(layer, 2, seed=3, zp_w="tensor")
    acc = oracle.conv2d_acc(c.x, c.zp_x, c.w, c.zp_w, c.bias, c.stride, c.pads)
    idx = W.sample_indices(acc.size, 3000, seed=4)
    pts = oracle.conv2d_acc_points(c.x, c.zp_x, c.w, idx, c.zp_w, c.bias, c.stride, c.pads)
    np.testing.assert_array_equal(pts, acc.reshape(-1)[idx])


@pytest.mark.parametrize("depthwise", [False, True])
def test_uint8_weights_match_float64_library(oracle, depthwise):
    """Asymmetric uint8 weights (zero points in [0, 255]): the oracle's
    accumulator equals float64 library convolution of (Q_x - zp_x) and
    (Q_w - zp_w) with zero padding (exact: every partial sum is an integer
    below 2^53), for stride, asymmetric padding and per-channel zero points."""
    rng = np.random.default_rng(41)
    C = 6
    K = C if depthwise else 5
    x = rng.integers(0, 256, size=(2, 9, 8, C), dtype=np.uint8)
    w = (rng.integers(0, 256, size=(3, 2, C), dtype=np.uint8) if depthwise
         else rng.integers(0, 256, size=(K, 3, 2, C), dtype=np.uint8))
    zp_w = rng.integers(0, 256, size=K).astype(np.int32)
    bias = rng.integers(-999, 1000, size=K).astype(np.int32)
    stride, pads = (2, 1), (1, 0, 2, 1)
    acc = oracle.conv2d_acc(x, 131, w, zp_w, bias, stride, pads, depthwise=depthwise)
    xt = torch.from_numpy(x.astype(np.float64) - 131).permute(0, 3, 1, 2)
    xt = F.pad(xt, (pads[1], pads[3], pads[0], pads[2]))
    if depthwise:
        wt = torch.from_numpy(w.astype(np.float64) - zp_w[None, None, :]).permute(2, 0, 1)[:, None]
        ref = F.conv2d(xt, wt, stride=stride, groups=C)
    else:
        wt = torch.from_numpy(w.astype(np.float64) - zp_w[:, None, None, None]).permute(0, 3, 1, 2)
        ref = F.conv2d(xt, wt, stride=stride)
    ref = ref.permute(0, 2, 3, 1).numpy() + bias
    np.testing.assert_array_equal(acc, ref.astype(np.int64))


def test_uint8_weights_dequantize_identity(oracle):
    """Eq. (1)/(2) with uint8 weights: the real conv of s_x(Q_x - zp_x) and
    s_w(Q_w - zp_w) (real 0.0 in the padding) equals s_x*s_w[k]*acc, exactly."""
    rng = np.random.default_rng(42)
    x = rng.integers(0, 256, size=(1, 4, 5, 2), dtype=np.uint8)
    w = rng.integers(0, 256, size=(3, 2, 2, 2), dtype=np.uint8)
    zp_w = [200, 3, 128]
    s_w = [float(np.float32(v)) for v in (0.01, 0.003, 0.02)]
    acc = oracle.conv2d_acc(x, 77, w, np.array(zp_w, np.int32), None, (1, 2), (1, 1, 0, 1))
    real = X.conv2d_real(x.tolist(), 0.05, 77, w.tolist(), s_w, zp_w, None, (1, 2), (1, 1, 0, 1))
    for idx in np.ndindex(acc.shape):
        assert real[idx[0]][idx[1]][idx[2]][idx[3]] == X.f32(0.05) * X.f32(s_w[idx[3]]) * int(acc[idx])


def test_uint8_weights_dense_brute_force(oracle):
    rng = np.random.default_rng(43)
    x = rng.integers(-128, 128, size=(3, 7), dtype=np.int8)
    w = rng.integers(0, 256, size=(4, 7), dtype=np.uint8)
    zp_w = np.array([0, 255, 128, 17], np.int32)
    acc = oracle.dense_acc(x, -5, w, zp_w, None)
    for m in range(3):
        for j in range(4):
            assert acc[m, j] == sum((int(x[m, k]) + 5) * (int(w[j, k]) - int(zp_w[j])) for k in range(7))
