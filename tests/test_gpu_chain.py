"""Networks chained as they run, on the GPU against the oracle running the
same chain on its own tensors, every intermediate tensor byte for byte:
ResNet-50's conv body (stem, max pool, the 16 bottleneck blocks with int8
hand-off and a qnn.add closing every block, global average pool: 71
steps); MobileNet-V2's 17 expansion-6 inverted residuals (1x1 expand,
depthwise 3x3, 1x1 project, residual qnn.add: 58 steps); Inception-v3's
Mixed 5b and 5c (four branches, average-pool branch, channel concat with
the block's common quantization: 16 steps).  The ResNet and MobileNet
chains also run with each residual add fused into the epilogue of the conv
that qualifies for it, wherever that conv's plan accepts it."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from gpu_util import Q, O, log, dev, assert_equal  # noqa: E402
from paper_2006_10226_amd.fusion import residual_fusions  # noqa: E402


def run_chain_gpu(ch, fuse=False):
    """Runs the chain; fuse: residual adds that a conv's plan accepts run in
    its epilogue (the conv's own output is then never written).  Returns
    the tensors and the number of fused adds."""
    t = {"x0": dev(ch.x0)}
    keep = []
    by_conv = {c: (i, r) for i, (c, r) in residual_fusions(ch.graph()).items()} if fuse else {}
    skip = set()
    for idx, st in enumerate(ch.steps):
        if idx in skip:
            continue
        if isinstance(st, W.ChainConv):
            s_x, zp_x = ch.q[st.src]
            L = st.layer
            w, b = dev(st.w), dev(st.bias)
            keep += [w, b]
            shape = tuple(t[st.src].shape)
            if L.depthwise:
                p = Q.depthwise_conv2d_plan(shape, "i8", s_x, zp_x, w, st.s_w, st.zp_w, b, L.stride, L.pads, 1,
                                            st.s_y, st.zp_y, "i8", st.act)
            elif st.y_off is not None:
                p = Q.conv2d_plan(shape, "i8", s_x, zp_x, w, st.s_w, st.zp_w, b, L.stride, L.pads, 1, st.s_y,
                                  st.zp_y, "i8", st.act, y_ldc=st.y_off[1], y_coff=st.y_off[0])
            else:
                p = Q.conv2d_plan(shape, "i8", s_x, zp_x, w, st.s_w, st.zp_w, b, L.stride, L.pads,
                                  1, st.s_y, st.zp_y, "i8", st.act)
            if idx in by_conv:
                ai, rname = by_conv[idx]
                add = ch.steps[ai]
                try:
                    p.set_residual("i8", *ch.q[rname], add.s_o, add.zp_o, "i8", act=add.act)
                except Q.QnnError:
                    pass
                else:
                    out = p.new_output()
                    p.run(t[st.src], out, residual=t[rname])
                    torch.cuda.synchronize()
                    log(f"fused {st.dst} + {rname} -> {add.dst}: {p.describe()}")
                    p.close()
                    t[add.dst] = out
                    skip.add(ai)
                    continue
            if st.y_off is not None and st.dst not in t:
                t[st.dst] = torch.full(p.y_ldc_shape, 77, dtype=torch.int8, device="cuda")
            out = t[st.dst] if st.y_off is not None else p.new_output()
            p.run(t[st.src], out)
            torch.cuda.synchronize()
            p.close()
            t[st.dst] = out
        elif isinstance(st, W.ChainPool):
            t[st.dst] = Q.pool2d(t[st.src], st.mode, st.kernel, st.stride, st.pads)
        else:
            s_a, zp_a = ch.q[st.a]
            s_b, zp_b = ch.q[st.b]
            t[st.dst] = Q.add(t[st.a], s_a, zp_a, t[st.b], s_b, zp_b, st.s_o, st.zp_o, "i8", st.act)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in t.items()}, len(skip)


def run_chain_oracle(ch):
    t = {"x0": ch.x0}
    for st in ch.steps:
        if isinstance(st, W.ChainConv):
            s_x, zp_x = ch.q[st.src]
            L = st.layer
            y = O.conv2d(t[st.src], s_x, zp_x, st.w, st.s_w, st.zp_w, st.bias, st.s_y, st.zp_y, "i8",
                         st.act, "half_up", stride=(L.stride, L.stride), pads=L.pads, depthwise=L.depthwise)
            if st.y_off is None:
                t[st.dst] = y
            else:
                off, total = st.y_off
                if st.dst not in t:
                    t[st.dst] = np.full(y.shape[:3] + (total,), 77, np.int8)
                t[st.dst][..., off:off + y.shape[3]] = y
        elif isinstance(st, W.ChainPool):
            t[st.dst] = O.pool2d(t[st.src], st.mode, st.kernel, st.stride, st.pads)
        else:
            s_a, zp_a = ch.q[st.a]
            s_b, zp_b = ch.q[st.b]
            t[st.dst] = O.add(t[st.a], s_a, zp_a, t[st.b], s_b, zp_b, st.s_o, st.zp_o, "i8", st.act)
    return t


def check_chain(ch, gpu, ref, fused, what):
    """Every tensor the GPU chain wrote equals the oracle's; with fused
    adds, only the fused convs' own outputs are missing."""
    missing = [st.dst for st in ch.steps if st.dst not in gpu]
    assert len(missing) == fused, missing
    for st in ch.steps:
        if st.dst in gpu:
            assert_equal(gpu[st.dst], ref[st.dst], f"{what} {st.dst}")


@pytest.mark.parametrize("fuse", [False, True])
@pytest.mark.parametrize("N", [1, 2])
def test_resnet50_chain(N, fuse):
    ch = W.resnet50_chain(N)
    log(f"chain N={N} fuse={fuse}: {len(ch.steps)} steps")
    gpu, fused = run_chain_gpu(ch, fuse)
    ref = run_chain_oracle(ch)
    log(f"  {fused} adds fused")
    check_chain(ch, gpu, ref, fused, f"chain N={N} fuse={fuse}")
    assert fuse or fused == 0
    assert len(ch.steps) == 71 and ch.steps[-1].dst == "gap" and ref["gap"].shape == (N, 1, 1, 2048)
    # the data stays informative through the chain: the last block output
    # and the pooled features are neither constant nor all on the clamp
    assert len(np.unique(ref[ch.steps[-2].dst])) > 50
    assert len(np.unique(ref["gap"])) > 20


@pytest.mark.parametrize("fuse", [False, True])
@pytest.mark.parametrize("N", [1, 2])
def test_mobilenet_v2_chain(N, fuse):
    ch = W.mobilenet_v2_chain(N)
    log(f"mobilenet chain N={N} fuse={fuse}: {len(ch.steps)} steps")
    gpu, fused = run_chain_gpu(ch, fuse)
    ref = run_chain_oracle(ch)
    log(f"  {fused} adds fused")
    check_chain(ch, gpu, ref, fused, f"mobilenet chain N={N} fuse={fuse}")
    assert len(ch.steps) == 58 and ref[ch.steps[-1].dst].shape == (N, 7, 7, 320)
    assert len(np.unique(ref[ch.steps[-1].dst])) > 50


@pytest.mark.parametrize("N", [1, 2])
def test_inception_mixed5_chain(N):
    ch = W.inception_v3_mixed5_chain(N)
    log(f"inception mixed chain N={N}: {len(ch.steps)} steps")
    gpu, fused = run_chain_gpu(ch, fuse=True)    # no residual adds: nothing to fuse
    ref = run_chain_oracle(ch)
    check_chain(ch, gpu, ref, fused, f"inception chain N={N}")
    assert fused == 0
    # every channel of both concats was written by a branch (no sentinel left)
    for g, total in (("mixed5b", 256), ("mixed5c", 288)):
        assert ref[g].shape == (N, 35, 35, total)
        assert not (gpu[g] == 77).all(axis=(0, 1, 2)).any(), g
    assert len(np.unique(ref["mixed5c"])) > 50


@pytest.mark.parametrize("workload,fn", [("resnet50_b32_chain", "resnet50_chain"),
                                         ("mobilenet_v2_b64_chain", "mobilenet_v2_chain"),
                                         ("inception_v3_mixed5_b64_chain", "inception_v3_mixed5_chain")])
def test_chain_as_benchmarked(workload, fn):
    """The chained workloads at their benchmark batch, set up and run
    exactly as bench.py times them (its plans, tensors and fused adds): every
    tensor the step writes, byte for byte, against the oracle's chain."""
    import bench
    t = {}
    items, N = bench.setup_chain(workload, fuse=True, tensors=t)
    for it in items:
        it.run()
    torch.cuda.synchronize()
    fused = sum(1 for it in items if getattr(it, "residual", None) is not None)
    log(f"{workload}: {len(items)} launches, {fused} adds fused")
    ch = getattr(W, fn)(N)
    ref = run_chain_oracle(ch)
    gpu = {k: v.cpu().numpy() for k, v in t.items()}
    check_chain(ch, gpu, ref, fused, workload)
    assert fused > 0 or fn == "inception_v3_mixed5_chain"   # Inception blocks have no residual adds
