"""GPU parity of conv2d / dense / depthwise + requantize: the HIP path (called
through the C ABI) against the CPU oracle, element by element, bit-exact."""
import zlib

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # the gpu marker deselects these on CPU hosts
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import (Q, O, log, dev, env, run_gpu, run_oracle, oracle_points, make_plan, assert_equal)  # noqa: E402


@pytest.mark.parametrize("s_y", [0.05, 0.5], ids=["sy0.05", "sy0.5"])
@pytest.mark.parametrize("one_shot", [False, True], ids=["plan", "oneshot"])
def test_single_conv_14x14x64(s_y, one_shot):
    c = W.single_conv_case(seed=1, s_y=s_y)
    log(f"single conv s_y={s_y} one_shot={one_shot}")
    assert_equal(run_gpu(c, one_shot), run_oracle(c), "conv14x14x64")


@pytest.mark.parametrize("layer,seed", [(W.bert_ffn()[0], 2), (W.bert_ffn()[1], 3)], ids=["768to3072", "3072to768"])
def test_dense_bert_ffn(layer, seed):
    c = W.dense_case(layer, seed)
    log(f"dense {layer}")
    assert_equal(run_gpu(c), run_oracle(c), layer.name)
    assert_equal(run_gpu(c, one_shot=True), run_oracle(c), layer.name + " one-shot")


def test_dense_two_stage_rounding():
    c = W.dense_case(W.bert_ffn()[0], 7)
    c.rounding = "two_stage"
    log("dense two-stage")
    assert_equal(run_gpu(c), run_oracle(c), "dense two-stage")


def test_resnet50_batch1_full():
    for i, layer in enumerate(W.resnet50()):
        c = W.conv_case(layer, 1, seed=3000 + i)
        log(f"resnet50 b1 {layer.name}")
        assert_equal(run_gpu(c), run_oracle(c), layer.name)


def test_resnet50_batch32_sampled():
    """The benchmark configuration (batch 32, the plans bench.py times),
    checked on sampled outputs."""
    for i, layer in enumerate(W.resnet50()):
        c = W.conv_case(layer, 32, seed=3000 + i)
        log(f"resnet50 b32 {layer.name}")
        p, keep = make_plan(c)
        y = p.run(dev(c.x)).cpu().numpy()
        p.close()
        idx = W.sample_indices(y.size, 3000, seed=i)
        assert_equal(y.reshape(-1)[idx], oracle_points(c, idx), layer.name)


def _mobilenet_cases(N):
    out = []
    for i, layer in enumerate(W.mobilenet_v2_layers()):
        if isinstance(layer, W.AddLayer):
            out.append(("add", layer, W.add_case(layer, N, seed=4000 + i)))
        else:
            out.append(("conv", layer, W.conv_case(layer, N, seed=4000 + i)))
    return out


def _check_add(case, sample=None):
    a, b = dev(case.a), dev(case.b)
    y = Q.add(a, case.s_a, case.zp_a, b, case.s_b, case.zp_b, case.s_o, case.zp_o, case.yt, case.act,
              case.rounding).cpu().numpy()
    ref = O.add(case.a, case.s_a, case.zp_a, case.b, case.s_b, case.zp_b, case.s_o, case.zp_o, case.yt, case.act,
                case.rounding)
    assert_equal(y, ref, case.name)


def test_mobilenet_v2_batch1_full():
    for kind, layer, c in _mobilenet_cases(1):
        log(f"mobilenet b1 {layer.name}")
        if kind == "add":
            _check_add(c)
        else:
            assert_equal(run_gpu(c), run_oracle(c), layer.name)


def test_mobilenet_v2_batch64_sampled():
    for kind, layer, c in _mobilenet_cases(64):
        log(f"mobilenet b64 {layer.name}")
        if kind == "add":
            _check_add(c)
            continue
        p, keep = make_plan(c)
        y = p.run(dev(c.x)).cpu().numpy()
        p.close()
        idx = W.sample_indices(y.size, 3000, seed=7)
        assert_equal(y.reshape(-1)[idx], oracle_points(c, idx), layer.name)


def _inception_groups():
    """Per concat group: the common output (s, zp) and the member layers."""
    groups = {}
    for i, layer in enumerate(W.inception_v3()):
        if layer.concat:
            groups.setdefault(layer.concat[0], []).append((i, layer))
    return groups


@pytest.mark.parametrize("N", [1, 64], ids=["b1_full", "b64_sampled"])
def test_inception_v3_concat_blocks(N):
    """Every branch writes its channel slice of the block output with the
    block's common (scale, zero point); channels no conv writes (the pooling
    branches) keep their sentinel value."""
    rng = np.random.default_rng(5)
    for g, members in _inception_groups().items():
        total = members[0][1].concat[2]
        s_y = float(np.float32(10 ** rng.uniform(-1.5, -0.5)))
        zp_y = int(rng.integers(0, 256))
        Ho = Wo = None
        cases = []
        for i, layer in members:
            c = W.conv_case(layer, N, seed=5000 + i, out_q=(s_y, zp_y))
            cases.append((i, layer, c))
        # output spatial size from the first member
        ho, wo = Q.out_hw(members[0][1].H, members[0][1].W, members[0][1].R, members[0][1].S,
                          members[0][1].stride, members[0][1].pads)
        out = torch.full((N, ho, wo, total), 77, dtype=torch.uint8, device="cuda")
        written = np.zeros(total, bool)
        refs = []
        for i, layer, c in cases:
            log(f"inception b{N} {layer.name} -> {g}[{layer.concat[1]}:+{layer.Cout}]")
            p, keep = make_plan(c, y_ldc=total, y_coff=layer.concat[1])
            p.run(dev(c.x), out=out)
            torch.cuda.synchronize()
            p.close()
            written[layer.concat[1]:layer.concat[1] + layer.Cout] = True
            refs.append((layer, c))
        y = out.cpu().numpy()
        assert (y[..., ~written] == 77).all(), g
        for layer, c in refs:
            sl = y[..., layer.concat[1]:layer.concat[1] + layer.Cout]
            if N == 1:
                assert_equal(sl, run_oracle(c), layer.name)
            else:
                flat = np.ascontiguousarray(sl).reshape(-1)
                idx = W.sample_indices(flat.size, 2000, seed=9)
                assert_equal(flat[idx], oracle_points(c, idx), layer.name)


def test_inception_v3_other_layers_batch1():
    for i, layer in enumerate(W.inception_v3()):
        if layer.concat:
            continue
        c = W.conv_case(layer, 1, seed=5000 + i)
        log(f"inception b1 {layer.name}")
        assert_equal(run_gpu(c), run_oracle(c), layer.name)


# ------------------------------------------------------------------ variants

VARIANTS = [
    # (name, layer, N, kwargs)
    ("zpw_tensor", W.ConvLayer("v", 9, 11, 32, 40, 3, 3, 1, (1, 1, 1, 1)), 2, dict(zp_w="tensor")),
    ("zpw_channel", W.ConvLayer("v", 13, 7, 48, 24, 3, 3, 2, (1, 0, 1, 2)), 3, dict(zp_w="channel")),
    ("zpw_channel_1x1", W.ConvLayer("v", 5, 5, 64, 100, 1, 1), 4, dict(zp_w="channel")),
    ("half_away", W.ConvLayer("v", 10, 10, 64, 64, 3, 3, 1, (1, 1, 1, 1)), 2, dict(rounding="half_away")),
    ("int8_x", W.ConvLayer("v", 10, 12, 32, 48, 3, 3, 1, (1, 1, 1, 1)), 2, dict(x_dtype="i8")),
    ("int8_y", W.ConvLayer("v", 10, 12, 32, 48, 3, 3, 1, (1, 1, 1, 1)), 2, dict(yt="i8")),
    ("int32_y", W.ConvLayer("v", 10, 12, 32, 48, 3, 3, 1, (1, 1, 1, 1)), 2, dict(yt="i32")),
    ("int32_y_zpw", W.ConvLayer("v", 8, 9, 16, 20, 3, 3, 2, (0, 1, 2, 0)), 2, dict(yt="i32", zp_w="channel")),
    ("no_bias_no_act", W.ConvLayer("v", 7, 7, 128, 130, 3, 3, 1, (1, 1, 1, 1)), 1, dict(bias=False, act=None)),
    ("ragged_cout", W.ConvLayer("v", 6, 6, 32, 37, 3, 3, 1, (1, 1, 1, 1)), 3, {}),
    ("cin3_stem", W.ConvLayer("v", 31, 29, 3, 64, 7, 7, 2, (3, 3, 3, 3)), 2, {}),
    ("cin24_1x1", W.ConvLayer("v", 14, 14, 24, 144, 1, 1), 2, {}),
    ("cin20", W.ConvLayer("v", 9, 9, 20, 36, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    ("cin5", W.ConvLayer("v", 9, 9, 5, 8, 3, 3, 1, (2, 2, 2, 2)), 2, dict(zp_w="channel")),
    ("one_pixel", W.ConvLayer("v", 1, 1, 64, 64, 1, 1), 1, {}),
    ("big_filter", W.ConvLayer("v", 7, 7, 32, 16, 7, 7, 1, (3, 3, 3, 3)), 1, {}),
    ("1x7", W.ConvLayer("v", 17, 17, 128, 128, 1, 7, 1, (0, 3, 0, 3)), 2, {}),
    ("7x1", W.ConvLayer("v", 17, 17, 128, 192, 7, 1, 1, (3, 0, 3, 0)), 2, {}),
    ("stride2_asym", W.ConvLayer("v", 16, 15, 64, 64, 3, 3, 2, (0, 0, 1, 1)), 2, {}),
    ("deep_J", W.ConvLayer("v", 7, 7, 512, 64, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    ("dw_zpw", W.ConvLayer("v", 12, 12, 32, 32, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, dict(zp_w="channel")),
    ("dw_s2_i8", W.ConvLayer("v", 13, 13, 24, 24, 3, 3, 2, (1, 1, 1, 1), depthwise=True), 2, dict(x_dtype="i8")),
    ("dw_odd_c", W.ConvLayer("v", 9, 9, 7, 7, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, {}),
    ("dw_5x5_i32", W.ConvLayer("v", 9, 9, 16, 16, 5, 5, 1, (2, 2, 2, 2), depthwise=True), 2, dict(yt="i32")),
    ("dw_half_away", W.ConvLayer("v", 8, 8, 64, 64, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2,
     dict(rounding="half_away")),
    # the two-stage rounding through every epilogue: the LDS-direct / tap
    # kernels (3x3, C % 64 == 0), the short 1x1 form, the gather kernel (C
    # not a multiple of 64), the dot-product depthwise kernel and the
    # general one, int8 and uint8 outputs
    ("two_stage", W.ConvLayer("v", 10, 10, 64, 64, 3, 3, 1, (1, 1, 1, 1)), 2, dict(rounding="two_stage")),
    ("two_stage_1x1_i8", W.ConvLayer("v", 9, 9, 256, 100, 1, 1), 3, dict(rounding="two_stage", yt="i8")),
    ("two_stage_gather", W.ConvLayer("v", 9, 9, 20, 36, 3, 3, 1, (1, 1, 1, 1)), 2, dict(rounding="two_stage")),
    ("two_stage_deep", W.ConvLayer("v", 7, 7, 512, 64, 3, 3, 1, (1, 1, 1, 1)), 2, dict(rounding="two_stage")),
    ("dw_two_stage", W.ConvLayer("v", 8, 8, 64, 64, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2,
     dict(rounding="two_stage")),
    ("dw_5x5_two_stage", W.ConvLayer("v", 9, 9, 16, 16, 5, 5, 1, (2, 2, 2, 2), depthwise=True), 2,
     dict(rounding="two_stage", yt="i8")),
]


@pytest.mark.parametrize("name,layer,N,kw", VARIANTS, ids=[v[0] for v in VARIANTS])
def test_conv_variants(name, layer, N, kw):
    c = W.conv_case(layer, N, seed=zlib.crc32(name.encode()) % 1000, **kw)
    log(f"variant {name}")
    assert_equal(run_gpu(c), run_oracle(c), name)


@pytest.mark.parametrize("tile", list(range(9)))
def test_every_tile(tile):
    """Each kernel instantiation (tile shape x gather width), forced, on
    ragged shapes that span several tiles, with several tiles per
    persistent workgroup."""
    layer = W.ConvLayer("t", 23, 21, 64, 200, 3, 3, 1, (1, 1, 1, 1))
    with env(QNN_TILE=tile):
        for kw in ({}, dict(zp_w="channel"), dict(yt="i32")):
            c = W.conv_case(layer, 2, seed=tile * 10, **kw)
            assert_equal(run_gpu(c), run_oracle(c), f"tile {tile} {kw}")
        c = W.conv_case(W.ConvLayer("t", 9, 9, 3, 70, 5, 5, 2, (2, 2, 2, 2)), 3, seed=1)
        assert_equal(run_gpu(c), run_oracle(c), f"tile {tile} channel-padded gather")
        c = W.conv_case(W.ConvLayer("t", 9, 9, 24, 70, 3, 3, 1, (1, 1, 1, 1)), 3, seed=2)
        assert_equal(run_gpu(c), run_oracle(c), f"tile {tile} 8-byte gather")
        c = W.conv_case(W.ConvLayer("t", 40, 40, 64, 96, 3, 3, 1, (1, 1, 1, 1)), 8, seed=3)
        assert_equal(run_gpu(c), run_oracle(c), f"tile {tile} many tiles per workgroup")


def test_random_shapes():
    rng = np.random.default_rng(123)
    for t in range(40):
        R, S = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        H, Wd = int(rng.integers(R, 20)), int(rng.integers(S, 20))
        C = int(rng.choice([1, 3, 4, 8, 16, 32, 48, 64, 96, 160, 256]))
        K = int(rng.integers(1, 300))
        st = int(rng.integers(1, 3))
        pads = tuple(int(v) for v in rng.integers(0, 3, size=4))
        layer = W.ConvLayer("r", H, Wd, C, K, R, S, st, pads)
        kw = dict(zp_w=str(rng.choice(["zero", "tensor", "channel"])),
                  rounding=str(rng.choice(["half_up", "half_away", "two_stage"])),
                  x_dtype=str(rng.choice(["u8", "i8"])), yt=str(rng.choice(["u8", "i8", "i32"])),
                  bias=bool(rng.integers(0, 2)))
        c = W.conv_case(layer, int(rng.integers(1, 4)), seed=t, **kw)
        log(f"random {t}: {layer} {kw}")
        assert_equal(run_gpu(c), run_oracle(c), f"random {t}")


def test_empty_batch_is_noop():
    c = W.single_conv_case()
    x = torch.empty((0, 14, 14, 64), dtype=torch.uint8, device="cuda")
    y = Q.conv2d(x, c.s_x, c.zp_x, dev(c.w), c.s_w, c.zp_w, None, 1, 1, 1, c.s_y, c.zp_y, "u8")
    assert y.shape == (0, 14, 14, 64)
    p, keep = make_plan(c, N=0)
    p.run(x)
    torch.cuda.synchronize()
    p.close()
    # a fused residual add on an empty batch: nothing to read or write either
    with env(QNN_DMA=0):
        p, keep = make_plan(c, N=0)
    p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
    y = p.run(x, residual=torch.empty((0, 14, 14, 64), dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert y.shape == (0, 14, 14, 64)
    p.close()


def test_plan_workspace_and_streams():
    """Two runs of one plan that needs a workspace (window sums of term 3)
    on two streams, each with its own workspace, give the oracle's result."""
    layer = W.ConvLayer("ws", 7, 7, 512, 512, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 2, seed=11, zp_w="channel")
    ref = run_oracle(c)
    p, keep = make_plan(c)
    assert p.workspace_size > 0, p.describe()
    x = dev(c.x)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    ws1 = torch.zeros(p.workspace_size, dtype=torch.uint8, device="cuda")
    ws2 = torch.zeros(p.workspace_size, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        y1 = p.run(x, workspace=ws1, stream=s1)
    with torch.cuda.stream(s2):
        y2 = p.run(x, workspace=ws2, stream=s2)
    torch.cuda.synchronize()
    assert_equal(y1.cpu().numpy(), ref, "stream 1")
    assert_equal(y2.cpu().numpy(), ref, "stream 2")
    p.close()


def test_accumulator_near_int32_bound():
    """Extreme values at the accumulator bound: all-255 activations with zero
    point 0, all -128 weights with zero point 127, J = 33000 taps, so the
    true accumulator is -255*255*J = -2145825000, just inside int32, while
    the folded terms of Eq. (3) individually stay in range only modulo 2^32."""
    layer = W.ConvLayer("ext", 2, 2, 33000, 8, 1, 1)
    c = W.conv_case(layer, 1, seed=1, yt="i32", bias=False, zp_w="tensor")
    c.x[:] = 255
    c.zp_x = 0
    c.w[:] = -128
    c.zp_w[:] = 127
    ref = run_oracle(c)
    assert int(ref.min()) == -255 * 255 * 33000
    assert_equal(run_gpu(c), ref, "extreme int32")
    c.yt = "u8"
    c.act = None
    c.s_y = 1.0
    assert_equal(run_gpu(c), run_oracle(c), "extreme u8")


@pytest.mark.parametrize("staged", [0, 1])
def test_channel_slice_partial_chunk(staged):
    """Output written into a channel slice whose width is not a multiple of
    16 (the staged epilogue's last 16-byte chunk is partial), with both the
    LDS-staged and the direct store path; channels outside the slice keep
    their sentinel."""
    layer = W.ConvLayer("slice", 11, 13, 32, 20, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 3, seed=21)
    with env(QNN_STAGED=staged):
        p, keep = make_plan(c, y_ldc=48, y_coff=16)
    out = torch.full((3, 11, 13, 48), 201, dtype=torch.uint8, device="cuda")
    p.run(dev(c.x), out=out)
    torch.cuda.synchronize()
    p.close()
    y = out.cpu().numpy()
    assert (y[..., :16] == 201).all() and (y[..., 36:] == 201).all()
    assert_equal(y[..., 16:36], run_oracle(c), f"slice staged={staged}")


# The tap-uniform kernels (C % 64 == 0): every configuration of the
# LDS-direct family (DmaTile) and of the register-staged family (TapTile),
# forced, on shapes with ragged channel and pixel tiles, padding on every
# side (the border-class correction), strides, int8 activations (no flip),
# zero points of 0 (no correction), weight zero points (term 3) and int32
# outputs.
TAP_SHAPES = [
    (W.ConvLayer("t", 23, 21, 64, 200, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    (W.ConvLayer("t", 23, 21, 64, 200, 3, 3, 1, (1, 1, 1, 1)), 2, dict(zp_w="channel")),
    (W.ConvLayer("t", 23, 21, 64, 200, 3, 3, 1, (1, 1, 1, 1)), 2, dict(yt="i32")),
    (W.ConvLayer("t", 16, 15, 128, 96, 3, 3, 2, (0, 0, 1, 1)), 3, dict(x_dtype="i8")),
    (W.ConvLayer("t", 17, 17, 128, 72, 1, 7, 1, (0, 3, 0, 3)), 2, dict(rounding="half_away")),
    (W.ConvLayer("t", 9, 9, 256, 300, 1, 1), 5, dict(yt="i8")),
    (W.ConvLayer("t", 40, 40, 64, 96, 3, 3, 1, (1, 1, 1, 1)), 8, {}),
]


# 1x1 convolutions with one to four K-steps (the short-reduction forms of
# the LDS-direct kernel): ragged pixels and channels, stride 2, padding,
# int8 input and output, term 3, int32 output
SHORT_SHAPES = [
    (W.ConvLayer("s", 9, 9, 64, 300, 1, 1), 5, {}),
    (W.ConvLayer("s", 9, 11, 128, 72, 1, 1, 2), 3, dict(yt="i8")),
    (W.ConvLayer("s", 7, 5, 256, 200, 1, 1), 4, dict(zp_w="channel")),
    (W.ConvLayer("s", 8, 8, 64, 96, 1, 1, 1, (1, 1, 1, 1)), 2, dict(x_dtype="i8")),
    (W.ConvLayer("s", 6, 6, 192, 64, 1, 1), 3, {}),
    (W.ConvLayer("s", 10, 10, 128, 130, 1, 1), 2, dict(yt="i32")),
    (W.ConvLayer("s", 28, 28, 64, 160, 1, 1), 4, {}),   # 75-150 tiles
]
# K-steps each LDS-direct configuration holds in its short form (0: ring);
# the last three are ring forms with two K-step groups per tile (the
# shapes above have 4, 9, 14 and 18 K-steps: odd counts leave the second
# group a step past the end)
DMA_SHORT_STAGES = [0] * 15 + [1, 1, 1, 1, 2, 2, 2, 2, 4, 4, 4] + [0, 0, 0]


@pytest.mark.parametrize("tile", list(range(len(DMA_SHORT_STAGES))))
def test_every_dma_tile(tile):
    short = DMA_SHORT_STAGES[tile]
    shapes = TAP_SHAPES if not short else [sh for sh in SHORT_SHAPES if (sh[0].Cin + 63) // 64 <= short]
    with env(QNN_DMA=tile):
        for i, (layer, N, kw) in enumerate(shapes):
            c = W.conv_case(layer, N, seed=100 + tile * 10 + i, **kw)
            p, keep = make_plan(c)
            assert p.describe().startswith("conv_dma"), p.describe()
            p.close()
            log(f"dma tile {tile} shape {i}")
            assert_equal(run_gpu(c), run_oracle(c), f"dma tile {tile} shape {i} {kw}")
        # zero point 0: no padding correction table
        c = W.conv_case(shapes[0][0], 2, seed=7)
        c.zp_x = 0
        assert_equal(run_gpu(c), run_oracle(c), f"dma tile {tile} zp_x 0")


@pytest.mark.parametrize("tile", [26, 27, 28])
def test_split_dma_tiles_skip_row_pair_stem(tile):
    """The two-group tiles step the activations by two K-steps; the row-pair
    walk of a 3-channel stem steps one row pair at a time, so a forced
    two-group tile is not used there and the plan takes its own choice."""
    layer = W.ConvLayer("stem", 30, 30, 3, 64, 7, 7, 2, (3, 3, 3, 3))
    c = W.conv_case(layer, 2, seed=tile)
    with env(QNN_DMA=tile):
        p, keep = make_plan(c)
        d = p.describe()
        p.close()
        assert "threads=512" not in d, d
        assert_equal(run_gpu(c), run_oracle(c), f"stem with dma {tile} forced")


@pytest.mark.parametrize("layer,tile", [
    (W.ConvLayer("slice3x3", 12, 13, 64, 72, 3, 3, 1, (1, 1, 1, 1)), 3),
    (W.ConvLayer("slice1x1", 12, 13, 64, 72, 1, 1), 15),
    (W.ConvLayer("slice1x1", 12, 13, 192, 72, 1, 1), 23),
], ids=["ring", "short1", "short4"])
@pytest.mark.parametrize("coff", [8, 64])
def test_dma_channel_slice_output(layer, tile, coff):
    """LDS-direct kernel writing a channel slice of a wider output (y_ldc,
    y_coff): 16-byte aligned rows take the staged whole-chunk stores, others
    the direct ones; bytes outside the slice stay untouched."""
    c = W.conv_case(layer, 3, seed=31)
    total = 160
    with env(QNN_DMA=tile):
        p, keep = make_plan(c, y_ldc=total, y_coff=coff)
        d = p.describe()
        assert d.startswith("conv_dma"), d
        out = torch.full((3, 12, 13, total), 77, dtype=torch.uint8, device="cuda")
        p.run(dev(c.x), out=out)
        torch.cuda.synchronize()
        p.close()
    y = out.cpu().numpy()
    log(f"dma slice coff={coff}: {d}")
    assert_equal(y[..., coff:coff + 72], run_oracle(c), f"dma slice {coff}")
    rest = np.ones(total, bool)
    rest[coff:coff + 72] = False
    assert (y[..., rest] == 77).all()


# 3x3 depthwise layers of the dot-product kernel: strides 1 and 2,
# asymmetric pads, row tails (Wo not a multiple of 4), int8 input and
# output, int32 output, weight zero points, half-away rounding (64-bit
# requantize), 8 to 144 channels
DW3_SHAPES = [
    (W.ConvLayer("d", 13, 11, 144, 144, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, {}),
    (W.ConvLayer("d", 14, 15, 96, 96, 3, 3, 2, (0, 0, 1, 1), depthwise=True), 3, dict(x_dtype="i8")),
    (W.ConvLayer("d", 9, 10, 8, 8, 3, 3, 1, (2, 1, 0, 1), depthwise=True), 2, dict(yt="i8")),
    (W.ConvLayer("d", 12, 12, 32, 32, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, dict(zp_w="channel")),
    (W.ConvLayer("d", 11, 9, 16, 16, 3, 3, 2, (1, 1, 1, 1), depthwise=True), 2, dict(yt="i32", zp_w="tensor")),
    (W.ConvLayer("d", 8, 7, 64, 64, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, dict(rounding="half_away")),
    (W.ConvLayer("d", 5, 5, 24, 24, 3, 3, 1, (0, 0, 0, 0), depthwise=True), 4, dict(act=None)),
    # rows of several 16-pixel segments with a ragged last one
    (W.ConvLayer("d", 6, 37, 40, 40, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, {}),
    (W.ConvLayer("d", 7, 75, 24, 24, 3, 3, 2, (1, 1, 1, 1), depthwise=True), 2, dict(x_dtype="i8", yt="i8")),
    # band kernel shapes: column tiles with a ragged last strip, stride 2
    # both ways, a two-column left pad with no right pad
    (W.ConvLayer("d", 10, 38, 32, 32, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, {}),
    (W.ConvLayer("d", 15, 33, 48, 48, 3, 3, 2, (1, 1, 1, 1), depthwise=True), 2, dict(zp_w="channel")),
    (W.ConvLayer("d", 9, 20, 16, 16, 3, 3, 1, (0, 2, 1, 0), depthwise=True), 3, dict(x_dtype="i8")),
    # wider channel counts: 128 and 192 channels, stride 1 and 2
    (W.ConvLayer("d", 10, 12, 128, 128, 3, 3, 1, (1, 1, 1, 1), depthwise=True), 2, {}),
    (W.ConvLayer("d", 13, 14, 192, 192, 3, 3, 2, (1, 1, 1, 1), depthwise=True), 2,
     dict(x_dtype="i8", zp_w="channel")),
]


# kernel forms of the 3x3 depthwise path: the register kernel with work
# items of 1, 2 and 4 strips; the LDS-tiled band kernel with one-row bands
# on 64-thread workgroups (several strips per thread), eight-row bands,
# and four-row bands in column tiles of one strip; and whatever the plan's
# timing picks
DW3_KERNELS = [
    ("seg1", dict(QNN_DWBAND=0, QNN_DW3T=1)),
    ("seg2", dict(QNN_DWBAND=0, QNN_DW3T=2)),
    ("seg4", dict(QNN_DWBAND=0, QNN_DW3T=4)),
    ("band_r1_t64", dict(QNN_DWRB=1, QNN_DWBT=64)),
    ("band_r8", dict(QNN_DWRB=8)),
    ("band_r4_ct1", dict(QNN_DWRB=4, QNN_DWCT=1)),
    ("timed", {}),
]


@pytest.mark.parametrize("kern", [k for k, _ in DW3_KERNELS])
@pytest.mark.parametrize("i", range(len(DW3_SHAPES)))
def test_depthwise3x3_dot4(i, kern):
    """The 3x3 depthwise kernels against the oracle, and the general
    depthwise kernel (QNN_DW3=0) on the same case.  The band kernel takes
    rows of a multiple of 16 bytes, and column tiles narrower than a row
    only with C % 16 == 0; on the other shapes the plan keeps the register
    kernel."""
    layer, N, kw = DW3_SHAPES[i]
    c = W.conv_case(layer, N, seed=600 + i, **kw)
    ref = run_oracle(c)
    cfg = dict(DW3_KERNELS)[kern]
    with env(**cfg):
        p, keep = make_plan(c)
        d = p.describe()
        p.close()
        band_ok = (layer.W * layer.Cin) % 16 == 0 and ("QNN_DWCT" not in cfg or layer.Cin % 16 == 0)
        if kern.startswith("seg"):
            assert d.startswith("depthwise dot4") and f"seg={kern[3:]}" in d, d
        elif kern.startswith("band") and band_ok:
            assert d.startswith("depthwise band") and f"rows={cfg['QNN_DWRB']}" in d, d
        elif kern.startswith("band"):
            assert d.startswith("depthwise dot4"), d
        log(f"dw3 shape {i} {kern}: {d}")
        assert_equal(run_gpu(c), ref, f"dw3 shape {i} {kern} {kw}")
    if kern == "seg1":
        with env(QNN_DW3=0):
            assert_equal(run_gpu(c), ref, f"dw general shape {i} {kw}")


def test_depthwise3x3_slices_and_unaligned_input():
    """Channel slices of a wider output (8-byte aligned rows take 8-byte
    stores, others byte stores) and an input view that is not 8-byte
    aligned (the general kernel takes over)."""
    layer = W.ConvLayer("dslice", 10, 9, 48, 48, 3, 3, 1, (1, 1, 1, 1), depthwise=True)
    c = W.conv_case(layer, 2, seed=77)
    ref = run_oracle(c)
    for coff, kcfg in ((0, dict(QNN_DWRB=2)), (5, dict(QNN_DWRB=2)), (16, dict(QNN_DWRB=4, QNN_DWCT=1)),
                       (2, dict(QNN_DWRB=4, QNN_DWCT=1)), (0, dict(QNN_DWBAND=0, QNN_DW3T=1)),
                       (5, dict(QNN_DWBAND=0, QNN_DW3T=1)), (16, dict(QNN_DWBAND=0, QNN_DW3T=4)),
                       (5, dict(QNN_DWBAND=0, QNN_DW3T=4))):
        total = 80
        with env(**kcfg):
            p, keep = make_plan(c, y_ldc=total, y_coff=coff)
        out = torch.full((2, 10, 9, total), 77, dtype=torch.uint8, device="cuda")
        p.run(dev(c.x), out=out)
        torch.cuda.synchronize()
        p.close()
        y = out.cpu().numpy()
        assert_equal(y[..., coff:coff + 48], ref, f"dw3 slice {coff} {kcfg}")
        rest = np.ones(total, bool)
        rest[coff:coff + 48] = False
        assert (y[..., rest] == 77).all()
    # x at an odd byte offset inside a larger buffer (the general kernel),
    # and 8 bytes past a 16-byte boundary (the register kernel)
    for shift in (3, 8):
        buf = torch.zeros(c.x.size + 16, dtype=torch.uint8, device="cuda")
        xv = buf[shift:shift + c.x.size].view(c.x.shape)
        xv.copy_(dev(c.x))
        p, keep = make_plan(c)
        y = p.run(xv)
        torch.cuda.synchronize()
        p.close()
        assert_equal(y.cpu().numpy(), ref, f"dw3 x at byte offset {shift}")


@pytest.mark.parametrize("tile", list(range(12)))
def test_every_tap_tile(tile):
    with env(QNN_TAP=tile):
        for i, (layer, N, kw) in enumerate(TAP_SHAPES):
            c = W.conv_case(layer, N, seed=200 + tile * 10 + i, **kw)
            p, keep = make_plan(c)
            d = p.describe()
            p.close()
            if not d.startswith("conv_tap"):
                continue   # K-step of this tile does not divide the channel count
            log(f"tap tile {tile} shape {i}")
            assert_equal(run_gpu(c), run_oracle(c), f"tap tile {tile} shape {i} {kw}")


@pytest.mark.parametrize("C,forced", [(64, "dma"), (128, "tap"), (20, "gather"), (64, "auto")])
def test_dilation(C, forced):
    """Dilated taps (Eq. (2) with the tap index scaled by the dilation)."""
    layer = W.ConvLayer("dil", 15, 13, C, 40, 3, 3, 1, (2, 1, 2, 3))
    c = W.conv_case(layer, 2, seed=C)
    cfg = {"dma": dict(QNN_DMA=0), "tap": dict(QNN_TAP=3), "gather": {}, "auto": {}}[forced]
    w, b = dev(c.w), dev(c.bias)
    with env(**cfg):
        p = Q.conv2d_plan(c.x.shape, "u8", c.s_x, c.zp_x, w, c.s_w, c.zp_w, b, 1, c.pads, (2, 2), c.s_y, c.zp_y,
                          c.yt, c.act, c.rounding)
    y = p.run(dev(c.x))
    torch.cuda.synchronize()
    log(f"dilation C={C} {forced}: {p.describe()}")
    p.close()
    ref = O.conv2d(c.x, c.s_x, c.zp_x, c.w, c.s_w, c.zp_w, c.bias, c.s_y, c.zp_y, c.yt, c.act, c.rounding,
                   (1, 1), c.pads, (2, 2))
    assert_equal(y.cpu().numpy(), ref, f"dilation C={C} {forced}")


def test_autotuned_choice_is_a_candidate_and_exact():
    """Default plans time several kernels on their own shape and keep one;
    whichever is kept, the bytes are the oracle's."""
    layer = W.ConvLayer("auto", 28, 28, 128, 128, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 4, seed=5)
    p, keep = make_plan(c)
    d = p.describe()
    p.close()
    assert "cands=" in d and int(d.split("cands=")[1].split()[0]) > 1, d
    assert_equal(run_gpu(c), run_oracle(c), d)


def test_tuning_file_reuses_the_timed_choice(tmp_path):
    """A timed kernel choice is appended to the kernel-choice file; a plan of
    the same shape created after re-reading the file takes it without
    timing and still computes the oracle's bytes."""
    f = tmp_path / "tune.txt"
    layer = W.ConvLayer("tuned", 14, 14, 256, 256, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 2, seed=17)
    Q.set_tuning_file(str(f))
    try:
        p, keep = make_plan(c)
        d1 = p.describe()
        p.close()
        lines = f.read_text().split("\n")
        assert len([ln for ln in lines if ln]) == 1, lines
        Q.set_tuning_file(str(f))
        p, keep = make_plan(c)
        d2 = p.describe()
        p.close()
        assert d1.split(" cands=")[0] == d2.split(" cands=")[0], (d1, d2)
        assert len([ln for ln in f.read_text().split("\n") if ln]) == 1
        assert_equal(run_gpu(c), run_oracle(c), d2)
    finally:
        Q.set_tuning_file(None)


@pytest.mark.parametrize("split", [1, 2, 4, 8])
def test_every_wave_split(split):
    """The wave-independent kernel with 1, 2, 4 and 8 waves sharing a tile's
    reduction, forced, on the tap-kernel shapes (ragged tiles, padding,
    strides, int8 input, term 3, int32 output, odd step counts)."""
    with env(QNN_WAVE=split):
        for i, (layer, N, kw) in enumerate(TAP_SHAPES):
            c = W.conv_case(layer, N, seed=300 + split * 10 + i, **kw)
            p, keep = make_plan(c)
            assert p.describe().startswith("conv_wave"), p.describe()
            p.close()
            log(f"wave split {split} shape {i}")
            assert_equal(run_gpu(c), run_oracle(c), f"wave split {split} shape {i} {kw}")
        c = W.conv_case(TAP_SHAPES[0][0], 2, seed=8)
        c.zp_x = 0
        assert_equal(run_gpu(c), run_oracle(c), f"wave split {split} zp_x 0")


@pytest.mark.parametrize("layer,N", [
    (W.ConvLayer("stem", 29, 31, 3, 64, 7, 7, 2, (3, 3, 3, 3)), 3),
    (W.ConvLayer("stem3", 35, 33, 3, 32, 3, 3, 2, (0, 0, 0, 0)), 2),
    (W.ConvLayer("stem3p", 20, 20, 3, 40, 3, 3, 1, (1, 2, 0, 1)), 2),
    (W.ConvLayer("stem4", 29, 32, 3, 64, 7, 7, 2, (3, 3, 3, 3)), 3),     # RGB rows of whole dwords
    (W.ConvLayer("stem4n", 10, 24, 3, 16, 3, 3, 1, (0, 0, 0, 0)), 2),    # padded rows wider than the image
    (W.ConvLayer("c8", 17, 16, 8, 24, 3, 3, 1, (1, 1, 1, 1)), 2),
    (W.ConvLayer("c4_5x5", 15, 15, 4, 70, 5, 5, 2, (2, 2, 2, 2)), 2),
    (W.ConvLayer("c1_5x5", 27, 27, 1, 20, 5, 5, 2, (2, 1, 2, 1)), 2),
    (W.ConvLayer("c2", 9, 40, 2, 72, 3, 3, 1, (1, 1, 1, 1)), 3),
])
def test_row_pair_mode(layer, N):
    """Small channel counts (S * C4 <= 32) through the row-pair mode of the
    LDS-direct kernel (zero-point padded image, two filter rows per
    K-step), for every configuration the plan may pick."""
    cfgs = [{}] + [dict(QNN_DMA=t) for t in (0, 3, 4, 12, 15, 19, 23, 24, 25)]
    for cfg in cfgs:
        for kw in ({}, dict(x_dtype="i8", yt="i8")):
            c = W.conv_case(layer, N, seed=17, **kw)
            with env(**cfg):
                p, keep = make_plan(c)
            d = p.describe()
            p.close()
            assert d.startswith("conv_dma"), d
            with env(**cfg):
                got = run_gpu(c)
            assert_equal(got, run_oracle(c), f"{layer.name} {cfg} {kw}: {d}")


# Stride-1 3x3 layers of the window kernel (conv_halo.hip), forced with 4
# and 8 waves per workgroup where its LDS fits: one and two 64-channel
# slices, whole-row tiles of 1 to 7 rows with a short last band, a 64-pixel
# row, ragged and several channel tiles, asymmetric and no padding, int8
# input and output, weight zero points, int32 output, half-away rounding.
HALO_SHAPES = [
    (W.ConvLayer("h56", 56, 56, 64, 64, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    (W.ConvLayer("h28", 28, 28, 128, 128, 3, 3, 1, (1, 1, 1, 1)), 2, {}),
    (W.ConvLayer("h13", 13, 13, 64, 96, 3, 3, 1, (1, 1, 1, 1)), 3, {}),
    (W.ConvLayer("h64", 9, 64, 64, 72, 3, 3, 1, (1, 1, 1, 1)), 2, dict(x_dtype="i8")),
    (W.ConvLayer("hpad", 12, 10, 64, 64, 3, 3, 1, (0, 2, 1, 0)), 3, dict(yt="i8")),
    (W.ConvLayer("hnopad", 10, 11, 128, 80, 3, 3, 1, (0, 0, 0, 0)), 2, dict(zp_w="channel")),
    (W.ConvLayer("h1", 1, 1, 64, 64, 3, 3, 1, (1, 1, 1, 1)), 4, dict(yt="i32")),
    (W.ConvLayer("h7", 7, 7, 64, 300, 3, 3, 1, (1, 1, 1, 1)), 3, dict(rounding="half_away")),
]


def _halo_lds(layer, nw):
    """LDS bytes of a window-kernel launch: resident weights (R*S*C/64
    fragments of 4 KB), 64 channel records, the workgroup's input window
    (nw bands of tr output rows plus 2 rows, Wo + 2 columns, 64 bytes per
    cell and channel slice, in 1 KB loads), whose space later holds a 64 x
    80 byte staging tile per wave."""
    pt, pl, pb, pr = layer.pads
    Ho, Wo = layer.H + pt + pb - 2, layer.W + pl + pr - 2
    tr = min(Ho, 64 // Wo)
    bands = -(-Ho // tr)
    rows = min(bands, nw) * tr + 2
    ninst = -(-(rows * (Wo + 2)) // 16)
    return 9 * layer.Cin // 64 * 4096 + 1024 + max(layer.Cin // 64 * ninst * 1024, nw * 64 * 80)


@pytest.mark.parametrize("nw", [4, 8])
def test_every_halo_config(nw):
    ran = 0
    seps = set()
    for i, (layer, N, kw) in enumerate(HALO_SHAPES):
        c = W.conv_case(layer, N, seed=700 + nw * 10 + i, **kw)
        with env(QNN_HALO=nw):
            p, keep = make_plan(c)
            d = p.describe()
            p.close()
            if not d.startswith("conv_halo"):
                assert _halo_lds(layer, nw) > 160 * 1024, d
                continue
            assert f"threads={nw * 64}" in d, d
            seps.add(d.split("sep=")[1].split()[0])
            log(f"halo nw {nw} shape {layer.name}: {d}")
            assert_equal(run_gpu(c), run_oracle(c), f"halo nw {nw} {layer.name} {kw}")
            ran += 1
    assert ran >= 5
    # both staging layouts: tiles in LDS of their own, tiles over the window
    assert seps == {"0", "1"}, seps
    # zero point 0: no padding correction table
    c = W.conv_case(HALO_SHAPES[2][0], 2, seed=9)
    c.zp_x = 0
    with env(QNN_HALO=nw):
        assert_equal(run_gpu(c), run_oracle(c), f"halo nw {nw} zp_x 0")


@pytest.mark.parametrize("coff", [8, 64])
def test_halo_channel_slice_output(coff):
    """Window kernel writing a channel slice of a wider output: staged
    16-byte chunks when aligned, direct stores otherwise; bytes outside the
    slice stay untouched."""
    layer = W.ConvLayer("hslice", 12, 13, 64, 72, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 3, seed=33)
    total = 160
    with env(QNN_HALO=8):
        p, keep = make_plan(c, y_ldc=total, y_coff=coff)
        d = p.describe()
        assert d.startswith("conv_halo"), d
        out = torch.full((3, 12, 13, total), 77, dtype=torch.uint8, device="cuda")
        p.run(dev(c.x), out=out)
        torch.cuda.synchronize()
        p.close()
    y = out.cpu().numpy()
    assert_equal(y[..., coff:coff + 72], run_oracle(c), f"halo slice {coff}")
    rest = np.ones(total, bool)
    rest[coff:coff + 72] = False
    assert (y[..., rest] == 77).all()


# Stride-1 3x3 layers of the streaming window kernel (conv_window.hip),
# every configuration forced where its LDS fits: bands shared within an
# image and whole-image bands (batch not a multiple of the bands per
# workgroup), one to eight channel slices (a partial last slice group),
# ragged and several channel tiles, asymmetric and no padding, int8 input
# and output, weight zero points, int32 output, half-away rounding.
WIN_SHAPES = [
    (W.ConvLayer("w14", 14, 14, 256, 256, 3, 3, 1, (1, 1, 1, 1)), 3, {}),
    (W.ConvLayer("w7", 7, 7, 512, 200, 3, 3, 1, (1, 1, 1, 1)), 5, {}),
    (W.ConvLayer("w13", 13, 13, 192, 96, 3, 3, 1, (1, 1, 1, 1)), 2, dict(x_dtype="i8")),
    (W.ConvLayer("wpad", 12, 10, 128, 64, 3, 3, 1, (0, 2, 1, 0)), 3, dict(yt="i8")),
    (W.ConvLayer("wnopad", 10, 11, 320, 80, 3, 3, 1, (0, 0, 0, 0)), 2, dict(zp_w="channel")),
    (W.ConvLayer("w1", 1, 1, 64, 48, 3, 3, 1, (1, 1, 1, 1)), 5, dict(yt="i32")),
    (W.ConvLayer("w28", 28, 28, 128, 40, 3, 3, 1, (1, 1, 1, 1)), 2, dict(rounding="half_away")),
]
WIN_CFGS = [(4, 2, 2), (2, 2, 2), (4, 1, 2), (8, 1, 2)]


def _win_lds(layer, cfg):
    """LDS bytes of a streaming-window launch: two weight groups (KS slices
    x 9 taps x TCB 1 KB fragments; the partial sums and 1 KB of channel
    records reuse them), the window (the staging tiles reuse it)."""
    nb, ks, tcb = WIN_CFGS[cfg]
    pt, pl, pb, pr = layer.pads
    Ho, Wo = layer.H + pt + pb - 2, layer.W + pl + pr - 2
    tr = min(Ho, 64 // Wo)
    bands = -(-Ho // tr)
    rows = nb * (Ho + 2) if bands == 1 else min(bands, nb) * tr + 2
    ninst = -(-(rows * (Wo + 2)) // 16)
    wgt = max(2 * tcb * ks * 9 * 1024, nb * (ks - 1) * tcb * 4 * 1024 + 1024)
    return wgt + max(layer.Cin // 64 * ninst * 1024, nb * 64 * (16 * tcb + 16))


@pytest.mark.parametrize("cfg", range(len(WIN_CFGS)))
def test_every_window_config(cfg):
    ran = 0
    for i, (layer, N, kw) in enumerate(WIN_SHAPES):
        c = W.conv_case(layer, N, seed=800 + cfg * 10 + i, **kw)
        with env(QNN_WIN=cfg):
            p, keep = make_plan(c)
            d = p.describe()
            p.close()
            if not d.startswith("conv_window"):
                assert _win_lds(layer, cfg) > 160 * 1024, d
                continue
            assert d.endswith(f"cfg={cfg}"), d
            log(f"window cfg {cfg} shape {layer.name}: {d}")
            assert_equal(run_gpu(c), run_oracle(c), f"window cfg {cfg} {layer.name} {kw}")
            ran += 1
    assert ran >= 4
    c = W.conv_case(WIN_SHAPES[2][0], 2, seed=10)
    c.zp_x = 0
    with env(QNN_WIN=cfg):
        assert_equal(run_gpu(c), run_oracle(c), f"window cfg {cfg} zp_x 0")


@pytest.mark.parametrize("coff", [8, 64])
def test_window_channel_slice_output(coff):
    """Streaming window kernel writing a channel slice of a wider output."""
    layer = W.ConvLayer("wslice", 12, 13, 128, 72, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 3, seed=34)
    total = 160
    with env(QNN_WIN=0):
        p, keep = make_plan(c, y_ldc=total, y_coff=coff)
        d = p.describe()
        assert d.startswith("conv_window"), d
        out = torch.full((3, 12, 13, total), 77, dtype=torch.uint8, device="cuda")
        p.run(dev(c.x), out=out)
        torch.cuda.synchronize()
        p.close()
    y = out.cpu().numpy()
    assert_equal(y[..., coff:coff + 72], run_oracle(c), f"window slice {coff}")
    rest = np.ones(total, bool)
    rest[coff:coff + 72] = False
    assert (y[..., rest] == 77).all()


# 1x1 convolutions whose channel count is a multiple of 16 but not of 64:
# the tap-walk kernels run them with a last K-step that reads past each
# pixel into the next ones (and past the end of x into out-of-range zeros),
# against zero weights.  Forced LDS-direct (ring and short forms) and
# register-staged tiles, plus the plan's own choice; stride 2, padding,
# int8 input and output, weight zero points, int32 output.
PARTIAL_1X1 = [
    (W.ConvLayer("p16", 9, 10, 16, 40, 1, 1), 3, {}),
    (W.ConvLayer("p48", 11, 9, 48, 72, 1, 1, 2), 2, dict(x_dtype="i8", yt="i8")),
    (W.ConvLayer("p80", 8, 8, 80, 200, 1, 1, 1, (1, 0, 0, 1)), 2, dict(zp_w="channel")),
    (W.ConvLayer("p144", 7, 9, 144, 24, 1, 1), 4, dict(yt="i32")),
    (W.ConvLayer("p160", 13, 6, 160, 96, 1, 1), 2, dict(rounding="half_away")),
    (W.ConvLayer("p208", 5, 5, 208, 130, 1, 1, 2, (1, 1, 1, 1)), 3, {}),
]


@pytest.mark.parametrize("forced", [{}, dict(QNN_DMA=0), dict(QNN_DMA=4), dict(QNN_DMA=12), dict(QNN_DMA=15),
                                    dict(QNN_DMA=23), dict(QNN_DMA=24), dict(QNN_TAP=0), dict(QNN_TAP=3),
                                    dict(QNN_TAP=7)],
                         ids=["auto", "dma0", "dma4", "dma12", "short1", "short4a", "short4b", "tap0", "tap3", "tap7"])
def test_one_by_one_partial_k_step(forced):
    for i, (layer, N, kw) in enumerate(PARTIAL_1X1):
        c = W.conv_case(layer, N, seed=900 + i, **kw)
        with env(**forced):
            p, keep = make_plan(c)
            d = p.describe()
            p.close()
            if "QNN_DMA" in forced:
                stages = DMA_SHORT_STAGES[forced["QNN_DMA"]]
                if stages and -(-layer.Cin // 64) > stages:
                    assert "cands=1 " not in d, d   # short form with fewer stages than K-steps: not forced
                    continue
                assert d.startswith("conv_dma"), d
            if "QNN_TAP" in forced:
                assert d.startswith("conv_tap"), d
            log(f"partial 1x1 {forced} {layer.name}: {d}")
            assert_equal(run_gpu(c), run_oracle(c), f"1x1 C={layer.Cin} {forced} {kw}: {d}")
