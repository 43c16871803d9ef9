"""Residual qnn.add fused into the conv epilogue (qnn_plan_set_residual,
qnn_plan_run_residual): byte-exact against the oracle's conv followed by
the oracle's qnn.add, for the kernel families that have the fused epilogue,
every dtype combination of the intermediate, the residual and the sum, both
rounding forms of the add, residual and output channel slices (16-byte and
byte paths), and the plans that must refuse it."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle as O
from gpu_util import Q, assert_equal, dev, env, log, make_plan, run_oracle

pytestmark = pytest.mark.gpu

# (layer, batch, forced kernel); 1x1 layers of the residual blocks and a 3x3
SHAPES = [
    (W.ConvLayer("b1x1", 9, 11, 64, 256, 1, 1, 1, (0, 0, 0, 0)), 2, dict(QNN_DMA=15)),
    (W.ConvLayer("b1x1t", 7, 9, 128, 96, 1, 1, 1, (0, 0, 0, 0)), 3, dict(QNN_TAP=1)),
    (W.ConvLayer("b3x3", 8, 10, 64, 80, 3, 3, 1, (1, 1, 1, 1)), 2, dict(QNN_DMA=0)),
    (W.ConvLayer("b1x1r", 6, 13, 64, 72, 1, 1, 1, (0, 0, 0, 0)), 2, dict(QNN_DMA=4)),
]


def _residual(shape, dtype, seed, r_ldc=None, r_coff=0):
    rng = np.random.default_rng(seed)
    N, Ho, Wo, K = shape
    r_ldc = K if r_ldc is None else r_ldc
    if dtype == "u8":
        full = rng.integers(0, 256, size=(N, Ho, Wo, r_ldc), dtype=np.uint8)
    else:
        full = rng.integers(-128, 128, size=(N, Ho, Wo, r_ldc), dtype=np.int8)
    return full, np.ascontiguousarray(full[..., r_coff:r_coff + K])


@pytest.mark.parametrize("i", range(len(SHAPES)))
@pytest.mark.parametrize("dts", [("u8", "u8", "u8"), ("i8", "i8", "i8"), ("u8", "i8", "i8"), ("i8", "u8", "u8")])
def test_fused_add_matches_conv_then_add(i, dts):
    layer, N, forced = SHAPES[i]
    yt, rt, ot = dts
    c = W.conv_case(layer, N, seed=900 + i, yt=yt)
    mid = run_oracle(c)                       # the conv output the plan computes (never stored when fused)
    for rounding, (s_r, s_o, zp_r, zp_o) in (("half_up", (0.031, 0.047, 7, -3 if ot == "i8" else 120)),
                                             ("half_away", (0.52, 0.011, -20 if rt == "i8" else 200, 5))):
        full, r = _residual(mid.shape, rt, seed=50 + i)
        act = (zp_o, 2 ** 31 - 1) if ot == "u8" else None     # ReLU on the sum (u8 outputs)
        ref = O.add(mid, c.s_y, c.zp_y, r, s_r, zp_r, s_o, zp_o, ot, act, rounding)
        y_ldc = -(-layer.Cout // 16) * 16          # fused outputs are stored as 16-byte rows
        with env(**forced):
            p, keep = make_plan(c, y_ldc=y_ldc)
        d = p.describe()
        assert d.startswith(("conv_dma", "conv_tap")), d
        p.set_residual(rt, s_r, zp_r, s_o, zp_o, ot, act=act, rounding=rounding)
        y = p.run(dev(c.x), residual=dev(full))
        torch.cuda.synchronize()
        log(f"fused add {layer.name} {dts} {rounding}: {p.describe()}")
        p.close()
        assert_equal(y.cpu().numpy()[..., :layer.Cout], ref, f"fused add {layer.name} {dts} {rounding}")


def test_fused_add_term_tables_and_without():
    """The epilogue adds through the plan's per-byte term tables wherever a
    32-bit sum of two terms cannot overflow, and through the add's own
    64-bit arithmetic where it can (a residual scale 10^7 times the
    output's); both byte-exact."""
    layer = W.ConvLayer("t1x1", 6, 9, 64, 64, 1, 1, 1, (0, 0, 0, 0))
    c = W.conv_case(layer, 2, seed=31)
    mid = run_oracle(c)
    for s_r, s_o, zp_r, zp_o, tables in ((0.02, 0.03, 130, 128, True), (4096.0, 0.0004096, 5, 100, False),
                                         (0.0004096, 4096.0, 250, 7, True)):
        full, r = _residual(mid.shape, "u8", seed=9)
        ref = O.add(mid, c.s_y, c.zp_y, r, s_r, zp_r, s_o, zp_o, "u8", None)
        with env(QNN_DMA=15):
            p, keep = make_plan(c)
        p.set_residual("u8", s_r, zp_r, s_o, zp_o, "u8")
        d = p.describe()
        assert d.endswith(" +add") == tables and d.endswith("+add(no-tables)") != tables, d
        y = p.run(dev(c.x), residual=dev(full))
        torch.cuda.synchronize()
        p.close()
        assert_equal(y.cpu().numpy(), ref, f"fused add scales {s_r} {s_o}: {d}")


@pytest.mark.parametrize("r_geom,y_geom", [((96, 16), (96, 0)), ((101, 5), (96, 16)), ((80, 0), (112, 32)),
                                            ((67, 3), (64, 0))])
def test_fused_add_slices(r_geom, y_geom):
    """Residual read from, and sum written to, channel slices of wider
    tensors: 16-byte aligned residual rows take the vector path, others the
    byte path; bytes outside the output slice stay untouched."""
    layer = W.ConvLayer("s1x1", 7, 9, 64, 64, 1, 1, 1, (0, 0, 0, 0))
    c = W.conv_case(layer, 2, seed=77)
    mid = run_oracle(c)
    r_ldc, r_coff = r_geom
    y_ldc, y_coff = y_geom
    full, r = _residual(mid.shape, "u8", seed=5, r_ldc=r_ldc, r_coff=r_coff)
    ref = O.add(mid, c.s_y, c.zp_y, r, 0.02, 130, 0.03, 128, "u8", None)
    with env(QNN_DMA=15):
        p, keep = make_plan(c, y_ldc=y_ldc, y_coff=y_coff)
    p.set_residual("u8", 0.02, 130, 0.03, 128, "u8", r_ldc=r_ldc, r_coff=r_coff)
    out = torch.full(mid.shape[:3] + (y_ldc,), 77, dtype=torch.uint8, device="cuda")
    p.run(dev(c.x), out=out, residual=dev(full))
    torch.cuda.synchronize()
    p.close()
    y = out.cpu().numpy()
    assert_equal(y[..., y_coff:y_coff + 64], ref, f"fused add slices {r_geom} {y_geom}")
    rest = np.ones(y_ldc, bool)
    rest[y_coff:y_coff + 64] = False
    assert (y[..., rest] == 77).all()


def test_fused_add_refused():
    """Plans without the fused epilogue refuse it and stay usable; a fused
    plan refuses a run without its residual."""
    layer = W.ConvLayer("r", 6, 7, 20, 32, 3, 3, 1, (1, 1, 1, 1))
    c = W.conv_case(layer, 2, seed=3)
    with env(QNN_TILE=0):                     # the gather kernel: no fused epilogue
        p, keep = make_plan(c)
    with pytest.raises(Q.QnnError, match="UNSUPPORTED"):
        p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
    assert_equal(p.run(dev(c.x)).cpu().numpy(), run_oracle(c), "refused plan still runs")
    p.close()
    c32 = W.conv_case(W.ConvLayer("r32", 6, 7, 64, 64, 1, 1, 1, (0, 0, 0, 0)), 2, seed=4, yt="i32")
    with env(QNN_DMA=15):
        p, keep = make_plan(c32)
    with pytest.raises(Q.QnnError, match="UNSUPPORTED"):
        p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
    p.close()
    c8 = W.conv_case(W.ConvLayer("r8", 6, 7, 64, 64, 1, 1, 1, (0, 0, 0, 0)), 2, seed=5)
    with env(QNN_DMA=15):
        p, keep = make_plan(c8)
    p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
    with pytest.raises(ValueError):
        p.run(dev(c8.x))                        # no residual
    # y not 16-byte aligned: refused before anything is enqueued
    shape = p.y_ldc_shape
    buf = torch.empty(int(np.prod(shape)) + 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(Q.QnnError, match="UNSUPPORTED"):
        p.run(dev(c8.x), out=buf[1:].view(shape), residual=torch.zeros(shape, dtype=torch.uint8, device="cuda"))
    p.close()
    # output rows that are not 16-byte multiples, and output not staged
    for kw, forced in ((dict(y_ldc=83, y_coff=3), dict(QNN_DMA=15)), ({}, dict(QNN_DMA=15, QNN_STAGED=0))):
        with env(**forced):
            p, keep = make_plan(c8, **kw)
        with pytest.raises(Q.QnnError, match="UNSUPPORTED"):
            p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
        p.close()


# LDS-direct and tap-walk configurations with a fused-add instantiation
# (waves of at most 64 x 64 outputs) and those without one.
DMA_FUSED = [t for t in range(29) if t not in (8, 9, 10, 11)]
DMA_SHORT = {t: s for t, s in zip(range(15, 26), [1, 1, 1, 1, 2, 2, 2, 2, 4, 4, 4])}
TAP_FUSED = list(range(8))


def _fused_case(layer, N, seed, env_kw, what, **kw):
    c = W.conv_case(layer, N, seed=seed, **kw)
    mid = run_oracle(c)
    full, r = _residual(mid.shape, "i8", seed=seed + 1)
    ref = O.add(mid, c.s_y, c.zp_y, r, 0.041, -9, 0.05, 3 if c.yt == "i8" else 110, c.yt, None)
    y_ldc = -(-layer.Cout // 16) * 16
    with env(**env_kw):
        p, keep = make_plan(c, y_ldc=y_ldc)
    d = p.describe()
    p.set_residual("i8", 0.041, -9, 0.05, 3 if c.yt == "i8" else 110, c.yt)
    with env(**env_kw):
        y = p.run(dev(c.x), residual=dev(full))
    torch.cuda.synchronize()
    p.close()
    log(f"fused {what}: {d}")
    assert_equal(y.cpu().numpy()[..., :layer.Cout], ref, f"fused {what}: {d}")
    return d


@pytest.mark.parametrize("tile", DMA_FUSED)
def test_fused_add_every_dma_tile(tile):
    """Every LDS-direct configuration that has the fused epilogue: a 1x1
    conv within its short form's K-steps (or a 3x3 conv with padding,
    int8 input and weight zero points for the ring forms), ragged channels
    and pixels."""
    if tile in DMA_SHORT:
        layer = W.ConvLayer("f1", 9, 11, 64 * DMA_SHORT[tile], 88, 1, 1)
        kw = {}
    else:
        layer = W.ConvLayer("f3", 10, 9, 64, 136, 3, 3, 1, (1, 1, 1, 1))
        kw = dict(x_dtype="i8", zp_w="channel", yt="i8")
    d = _fused_case(layer, 3, 500 + tile, dict(QNN_DMA=tile), f"dma {tile}", **kw)
    assert d.startswith("conv_dma"), d


@pytest.mark.parametrize("tile", TAP_FUSED)
def test_fused_add_every_tap_tile(tile):
    layer = W.ConvLayer("t3", 11, 10, 128, 100, 3, 3, 1, (1, 1, 1, 1))
    d = _fused_case(layer, 2, 600 + tile, dict(QNN_TAP=tile), f"tap {tile}", yt="i8")
    assert d.startswith("conv_tap"), d


@pytest.mark.parametrize("fam,tile", [("QNN_DMA", 8), ("QNN_DMA", 9), ("QNN_DMA", 10), ("QNN_DMA", 11),
                                      ("QNN_TAP", 8), ("QNN_TAP", 9), ("QNN_TAP", 10), ("QNN_TAP", 11)])
def test_fused_add_refused_for_large_wave_tiles(fam, tile):
    """Configurations whose waves hold more than 64 x 64 outputs have no
    fused epilogue: the plan refuses the add and runs as before."""
    layer = W.ConvLayer("b", 8, 8, 128, 128, 1, 1)
    c = W.conv_case(layer, 4, seed=tile)
    with env(**{fam: tile}):
        p, keep = make_plan(c)
    with pytest.raises(Q.QnnError, match="UNSUPPORTED"):
        p.set_residual("u8", 0.02, 10, 0.03, 5, "u8")
    assert_equal(p.run(dev(c.x)).cpu().numpy(), run_oracle(c), f"{fam}={tile} refused plan still runs")
    p.close()
