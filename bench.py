"""Benchmark of the quantized conv2d + requantize path on one MI355X.

Default workload: the ResNet-50 conv stack at batch 32 (stem, 16 bottlenecks,
4 projection shortcuts: 53 conv2d + bias + requantize (+ReLU) layers, NHWC
uint8 activations with random zero points, per-channel int8 weights), seeded
synthetic data.  A step runs every layer once on its own resident input;
the step is captured once into a HIP graph and replayed.

Printed (stdout, one JSON line): effective int8 TOP/s = 2 * algorithmic MACs
of the step / step time (MACs = N*Ho*Wo*Cout*R*S*Cin, zero-point corrections,
padding of the GEMM shape and the epilogue not counted), the roofline of the
dominant kernel, and the CPU oracle timed on a bounded sample.

Other workloads (--workload): mobilenet_v2_b64, inception_v3_b64, dense_bert,
conv14x14x64 -- the same measurement on those layer sets (depthwise layers
and adds are reported in GB/s in the per-layer file).  Chained networks,
each step reading the int8 tensor its producer wrote, TOP/s over the convs'
MACs and the whole chain's time: resnet50_b32_chain / resnet50_b1_chain
(ResNet-50's conv body: the stem, its max pool, the 16 bottleneck blocks
with a qnn.add closing each, the global average pool; 53 convs, 16 adds, 2
pools), mobilenet_v2_b64_chain / mobilenet_v2_b1_chain (the 17 inverted
residuals: 51 convs incl. 17 depthwise, 10 adds),
inception_v3_mixed5_b64_chain / inception_v3_mixed5_b1_chain (Mixed 5b and
5c: 14 convs, 2 average pools, channel concats).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Committed kernel choices (qnn_set_tuning_file records): the plans of these
# workloads take them instead of timing candidates on the machine at hand,
# so the benchmark and its profiles (and, for ResNet-50 b32, the
# full-tensor parity test of the same layers) run the same kernels.
CHOICE_FILES = {"resnet50_b32": os.path.join("workloads", "choices", "resnet50_b32.txt"),
                "mobilenet_v2_b64": os.path.join("workloads", "choices", "mobilenet_v2_b64.txt")}

PEAK_INT8_TOPS = 5000.0   # MI355X dense int8 MFMA, TOP/s
PEAK_HBM_GBS = 8000.0     # MI355X HBM3E, GB/s
METRIC = "effective int8 TOPS + % of int8 MFMA peak, qnn.conv2d+requantize"


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------ workloads

def _layers(name):
    import workloads as W
    if name == "resnet50_b32":
        return [("conv", l, W.conv_case(l, 32, seed=3000 + i)) for i, l in enumerate(W.resnet50())], 32
    if name == "resnet50_b1":
        return [("conv", l, W.conv_case(l, 1, seed=3000 + i)) for i, l in enumerate(W.resnet50())], 1
    if name == "mobilenet_v2_b64":
        out = []
        for i, l in enumerate(W.mobilenet_v2_layers()):
            if isinstance(l, W.AddLayer):
                out.append(("add", l, W.add_case(l, 64, seed=4000 + i)))
            else:
                out.append(("dw" if l.depthwise else "conv", l, W.conv_case(l, 64, seed=4000 + i)))
        return out, 64
    if name == "inception_v3_b64":
        return [("conv", l, W.conv_case(l, 64, seed=5000 + i)) for i, l in enumerate(W.inception_v3())], 64
    if name == "dense_bert":
        return [("dense", l, W.dense_case(l, seed=2 + i)) for i, l in enumerate(W.bert_ffn())], 128
    if name == "conv14x14x64":
        c = W.single_conv_case()
        return [("conv", W.SINGLE_CONV, c)], 1
    raise SystemExit(f"unknown workload {name}")


def _macs(kind, layer, case, out_shape):
    if kind == "dense":
        return layer.M * layer.K * layer.N
    if kind == "add":
        return 0
    N, Ho, Wo, K = out_shape
    if kind == "dw":
        return N * Ho * Wo * K * layer.R * layer.S
    return N * Ho * Wo * K * layer.R * layer.S * layer.Cin


def _bytes(kind, layer, case, out_shape):
    """Algorithmic HBM bytes: every input byte once, weights once, every
    output byte once."""
    if kind == "add":
        return case.a.nbytes * 3
    out = int(np.prod(out_shape))
    return case.x.nbytes + case.w.nbytes + out


class Item:
    pass


CHAINS = {
    "resnet50_b32_chain": ("resnet50_chain", 32),
    "resnet50_b1_chain": ("resnet50_chain", 1),
    "mobilenet_v2_b64_chain": ("mobilenet_v2_chain", 64),
    "mobilenet_v2_b1_chain": ("mobilenet_v2_chain", 1),
    "inception_v3_mixed5_b64_chain": ("inception_v3_mixed5_chain", 64),
    "inception_v3_mixed5_b1_chain": ("inception_v3_mixed5_chain", 1),
}


def setup_chain(workload, fuse=True, tensors=None):
    """Plans and device tensors of a chained network: every step writes its
    own output tensor (or its channel slice of a concat), which its
    consumers read.  fuse: each residual add that a conv's plan can run in
    its epilogue (paper_2006_10226_amd.fusion) runs there, and the conv's
    own output is never written.  tensors: a dict that receives the chain's
    device tensors by name (for tests)."""
    import torch
    import workloads as W
    from paper_2006_10226_amd import qnn as Q
    from paper_2006_10226_amd.fusion import residual_fusions

    fn, N = CHAINS[workload]
    ch = getattr(W, fn)(N)
    t = {"x0": torch.from_numpy(ch.x0).cuda()}
    fusions = residual_fusions(ch.graph()) if fuse else {}
    by_conv = {c: (i, r) for i, (c, r) in fusions.items()}
    skip = set()
    items = []
    for idx, st in enumerate(ch.steps):
        if idx in skip:
            continue
        it = Item()
        if isinstance(st, W.ChainConv):
            L = st.layer
            s_x, zp_x = ch.q[st.src]
            it.kind, it.layer, it.name = "conv", L, L.name
            it.w, it.bias = torch.from_numpy(st.w).cuda(), torch.from_numpy(st.bias).cuda()
            shape = tuple(t[st.src].shape)
            if L.depthwise:
                it.kind = "dw"
                it.plan = Q.depthwise_conv2d_plan(shape, "i8", s_x, zp_x, it.w, st.s_w, st.zp_w, it.bias, L.stride,
                                                  L.pads, 1, st.s_y, st.zp_y, "i8", st.act)
            else:
                off, total = st.y_off if st.y_off is not None else (0, None)
                it.plan = Q.conv2d_plan(shape, "i8", s_x, zp_x, it.w, st.s_w, st.zp_w, it.bias,
                                        L.stride, L.pads, 1, st.s_y, st.zp_y, "i8", st.act, y_ldc=total, y_coff=off)
            it.x = t[st.src]
            it.residual = None
            if idx in by_conv:
                ai, rname = by_conv[idx]
                add = ch.steps[ai]
                s_r, zp_r = ch.q[rname]
                try:
                    it.plan.set_residual("i8", s_r, zp_r, add.s_o, add.zp_o, "i8", act=add.act)
                    it.residual, skip_add = t[rname], ai
                    it.name = f"{L.name}+{add.name}"
                except Q.QnnError:
                    pass   # this plan's kernel has no fused epilogue: the add runs on its own
            if it.residual is not None:
                it.out = t[ch.steps[skip_add].dst] = it.plan.new_output()
                skip.add(skip_add)
            elif st.y_off is not None and st.dst in t:
                it.out = t[st.dst]   # another branch's slice of the same concat
            else:
                it.out = t[st.dst] = it.plan.new_output()
            it.desc = it.plan.describe()
            Nb, Ho, Wo, K = it.plan.out_shape
            it.macs = Nb * Ho * Wo * K * L.R * L.S * (1 if L.depthwise else L.Cin)
            it.bytes = it.x.numel() + st.w.size + Nb * Ho * Wo * K * (1 if it.residual is None else 2)
            if it.residual is None:
                it.run = (lambda it=it: it.plan.run(it.x, it.out))
            else:
                it.run = (lambda it=it: it.plan.run(it.x, it.out, residual=it.residual))
        elif isinstance(st, W.ChainPool):
            it.kind, it.layer, it.name, it.desc = "pool", None, st.name, "pool"
            it.x = t[st.src]
            it.args = (st.mode, st.kernel, st.stride, st.pads)
            it.out = t[st.dst] = Q.pool2d(it.x, *it.args)
            it.macs, it.bytes = 0, it.x.numel() + it.out.numel()
            it.run = (lambda it=it: Q.pool2d(it.x, *it.args, out=it.out))
        else:
            s_a, zp_a = ch.q[st.a]
            s_b, zp_b = ch.q[st.b]
            it.kind, it.layer, it.name, it.desc = "add", None, st.name, "add"
            it.a, it.b = t[st.a], t[st.b]
            it.out = t[st.dst] = torch.empty_like(it.a)
            it.args = (s_a, zp_a, s_b, zp_b, st.s_o, st.zp_o, st.act)
            it.macs, it.bytes = 0, 3 * it.a.numel()
            it.run = (lambda it=it: Q.add(it.a, it.args[0], it.args[1], it.b, it.args[2], it.args[3], it.args[4],
                                          it.args[5], "i8", it.args[6], out=it.out))
        items.append(it)
    if tensors is not None:
        tensors.update(t)
    return items, N


def setup(workload, fuse=True):
    import torch
    from paper_2006_10226_amd import qnn as Q

    if workload in CHAINS:
        return setup_chain(workload, fuse)
    layers, batch = _layers(workload)
    items = []
    for kind, layer, c in layers:
        it = Item()
        it.kind, it.layer, it.name = kind, layer, layer.name
        if kind == "add":
            it.a = torch.from_numpy(c.a).cuda()
            it.b = torch.from_numpy(c.b).cuda()
            it.out = torch.empty_like(it.a)
            it.case = c
            it.desc = "add"
            it.macs, it.bytes = 0, _bytes(kind, layer, c, None)
            it.run = (lambda it=it: Q.add(it.a, it.case.s_a, it.case.zp_a, it.b, it.case.s_b, it.case.zp_b,
                                          it.case.s_o, it.case.zp_o, "u8", out=it.out))
        else:
            w = torch.from_numpy(c.w).cuda()
            bias = None if c.bias is None else torch.from_numpy(c.bias).cuda()
            xdt = "u8" if c.x.dtype == np.uint8 else "i8"
            if kind == "dense":
                plan = Q.dense_plan(layer.M, layer.K, xdt, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.s_y, c.zp_y,
                                    c.yt, c.act, c.rounding)
            elif kind == "dw":
                plan = Q.depthwise_conv2d_plan(c.x.shape, xdt, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride,
                                               c.pads, 1, c.s_y, c.zp_y, c.yt, c.act, c.rounding)
            else:
                plan = Q.conv2d_plan(c.x.shape, xdt, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride, c.pads, 1,
                                     c.s_y, c.zp_y, c.yt, c.act, c.rounding)
            it.plan, it.w, it.bias = plan, w, bias
            it.x = torch.from_numpy(c.x).cuda()
            it.out = plan.new_output()
            it.ws = (torch.zeros(plan.workspace_size, dtype=torch.uint8, device="cuda")
                     if plan.workspace_size else None)
            it.desc = plan.describe()
            it.macs = _macs(kind, layer, c, plan.out_shape)
            it.bytes = _bytes(kind, layer, c, plan.out_shape)
            it.run = (lambda it=it: it.plan.run(it.x, it.out, it.ws))
        items.append(it)
        del c
    return items, batch


def kernel_group(it):
    """Kernel instantiation a layer runs (tile shape and gather width)."""
    if it.kind in ("add", "pool"):
        return it.kind
    if it.kind == "dw":
        return "depthwise"
    words = it.desc.split()
    d = dict(kv.split("=") for kv in words[1:] if "=" in kv)
    extra = f"gather={d['gather']}" if "gather" in d else f"threads={d['threads']} stages={d.get('stages', '')}"
    if "split" in d:
        extra += f" split={d['split']}"
    if "cfg" in d:
        extra += f" cfg={d['cfg']}"
    if "ksplit" in d:
        extra += " ksplit"
    if getattr(it, "residual", None) is not None:
        extra += " +add"
    return f"{words[0]} tile={d['tile']} {extra}"


# ------------------------------------------------------------------ timing

def time_steps(items, steps, warmup, use_graph):
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        for it in items:
            it.run()
    torch.cuda.synchronize()
    graph = None
    if use_graph:
        try:
            graph = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(stream)
            with torch.cuda.stream(s):
                with torch.cuda.graph(graph, stream=s):
                    for it in items:
                        it.run()
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
        except Exception as e:  # capture not possible: time eager launches
            log(f"graph capture failed ({e}); timing eager launches")
            graph = None
            torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        if graph is not None:
            graph.replay()
        else:
            for it in items:
                it.run()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps, graph


def _timed_plan(it):
    """Whether a step runs through qnn_plan_run_timed (plans without a fused add)."""
    return (getattr(it, "plan", None) is not None and it.kind in ("conv", "dense", "dw")
            and getattr(it, "residual", None) is None)


def time_launches(items, steps):
    """Per-launch kernel time over `steps` eager steps, on the stream the
    kernels run on (torch's current stream).  A layer with a plan runs through
    qnn_plan_run_timed, whose main kernel records the two events at its own
    start and end (hipExtLaunchKernel): its duration as rocprofv3 reports it.
    Other steps (adds, pools) ask the library to have their kernel record
    the events the same way (qnn_time_next_kernel).  Returns (median ms per
    item, how it was timed)."""
    import torch
    from paper_2006_10226_amd import qnn as Q
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in items]
          for _ in range(steps)]
    torch.cuda.synchronize()
    for s in range(steps):
        for i, it in enumerate(items):
            a, b = ev[s][i]
            if _timed_plan(it):
                it.plan.run_timed(it.x, it.out, getattr(it, "ws", None), a, b)
            else:
                Q.time_next_kernel(a, b)   # the kernel itself records them (add, pool, fused conv + add)
                it.run()
    torch.cuda.synchronize()
    per = np.array([[a.elapsed_time(b) for a, b in row] for row in ev])  # ms
    return np.median(per, axis=0), ["kernel"] * len(items)


def time_warm(items, reps=10):
    """Per-layer kernel time with the layer's inputs, weights and output
    already in the caches: each layer runs `reps` times back to back (after
    two untimed runs), timed by its own kernel's events as in
    time_launches.  Returns the median ms per item."""
    import torch
    from paper_2006_10226_amd import qnn as Q
    out = []
    for it in items:
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        it.run()
        it.run()
        for a, b in ev:
            if _timed_plan(it):
                it.plan.run_timed(it.x, it.out, getattr(it, "ws", None), a, b)
            else:
                Q.time_next_kernel(a, b)
                it.run()
        torch.cuda.synchronize()
        out.append(float(np.median([a.elapsed_time(b) for a, b in ev])))
    return np.array(out)


def library_gemm(items, reps=20):
    """A reference point beside the product, not part of it: the vendor's
    int8 GEMM (torch._int_mm, hipBLASLt on ROCm) on each conv or dense
    layer's GEMM shape (M output pixels x K channels x J = R*S*C, J rounded
    up to a multiple of 8 as the library requires), int32 output, without
    the gather, zero-point terms or requantize; `reps` calls back to back,
    replayed from a graph, caches warm.  Returns ms per item (nan for
    steps that are no GEMM)."""
    import torch
    out = []
    for it in items:
        if it.kind not in ("conv", "dense") or not it.macs:
            out.append(float("nan"))
            continue
        if it.kind == "dense":
            M, K = it.layer.M, it.layer.N
        else:
            Nb, Ho, Wo, K = it.plan.out_shape
            M = Nb * Ho * Wo
        J = -(-(it.macs // (M * K)) // 8) * 8
        a = torch.randint(-128, 128, (M, J), dtype=torch.int8, device="cuda")
        b = torch.randint(-128, 128, (K, J), dtype=torch.int8, device="cuda").t()   # column-major J x K
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            torch._int_mm(a, b)
            torch._int_mm(a, b)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(reps):
                torch._int_mm(a, b)
        g.replay()
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / reps)
        out.append(float(np.median(ts)))
        del g, a, b
    return np.array(out)


def sample_clock(items, graph_step, seconds=2.0, settle=1.0):
    """The GPU's graphics clock while the step runs: steps run back to back
    for `seconds` while a thread reads the current clock (amdsmi, through
    torch.cuda.clock_rate) every 10 ms.  The reading is refreshed by the
    driver only every 1/6 to 1 s, so only reads taken after `settle`
    seconds of stepping count.  Kept out of the timed steps so that the
    reads cannot slow their launches.  Returns {min, median, max, samples}
    in MHz, or None when the clock cannot be read."""
    import threading
    import torch
    try:
        torch.cuda.clock_rate()
    except Exception as e:   # no amdsmi on this machine: report no clock
        log(f"GPU clock not readable ({e})")
        return None
    reads, stop = [], threading.Event()
    t0 = time.perf_counter()

    def poll():
        while not stop.is_set():
            try:
                reads.append((time.perf_counter() - t0, int(torch.cuda.clock_rate())))
            except Exception:
                return
            time.sleep(0.01)

    th = threading.Thread(target=poll, daemon=True)
    th.start()
    try:
        while time.perf_counter() - t0 < seconds:
            for _ in range(10):
                if graph_step is not None:
                    graph_step.replay()
                else:
                    for it in items:
                        it.run()
            torch.cuda.synchronize()
    finally:
        stop.set()
        th.join()
    mhz = [m for t, m in reads if settle <= t <= seconds]
    if not mhz:
        return None
    return {"min": min(mhz), "median": int(np.median(mhz)), "max": max(mhz), "samples": len(mhz)}


# ------------------------------------------------------------------ CPU oracle baseline

def cpu_baseline(workload, target_s=12.0):
    """The oracle (plain int64 loop nests) on a bounded sample of the same
    layers: a fixed number of randomly chosen outputs per layer."""
    from oracle import oracle as O
    import workloads as W

    if workload in CHAINS:
        # the chain's conv shapes, sampled on independent seeded inputs
        fn, N = CHAINS[workload]
        ch = getattr(W, fn)(N)
        layers = [("dw" if st.layer.depthwise else "conv", st.layer, W.conv_case(st.layer, N, seed=7000 + i))
                  for i, st in enumerate(ch.steps) if isinstance(st, W.ChainConv)]
    else:
        layers, _ = _layers(workload)
    convs = [(k, l, c) for k, l, c in layers if k in ("conv", "dense", "dw")]

    def run(per_layer):
        macs = 0
        t0 = time.perf_counter()
        for i, (kind, layer, c) in enumerate(convs):
            if kind == "dense":
                rows = max(1, per_layer // layer.N)
                xs = c.x[:rows]
                O.dense_acc(xs, c.zp_x, c.w, c.zp_w, c.bias)
                macs += rows * layer.N * layer.K
                continue
            Ho, Wo = O.conv_out_hw(layer.H, layer.W, layer.R, layer.S, c.stride, c.pads)
            total = c.x.shape[0] * Ho * Wo * c.K
            idx = W.sample_indices(total, per_layer, seed=i)
            acc = O.conv2d_acc_points(c.x, c.zp_x, c.w, idx, c.zp_w, c.bias, c.stride, c.pads, (1, 1),
                                      c.depthwise)
            O.requantize_points(acc, idx, c.K, c.s_x, c.s_w, c.s_y, c.zp_y, c.yt, c.act, c.rounding)
            macs += idx.size * c.J
        return macs, time.perf_counter() - t0

    def grow(target):
        # grow the sample until one pass takes about `target` s of wall-clock
        per = 16
        while True:
            macs, t = run(per)
            if t >= 0.6 * target or per >= 4000000:
                return per, macs, t
            per = min(4000000, int(per * min(16.0, max(2.0, target / max(t, 1e-3)))))

    def sample(per, macs, t):
        return (f"{per} randomly chosen outputs of each of the {len(convs)} layers of the same workload "
                f"({macs / 1e9:.2f} G MAC in {t:.1f} s, requantize included)")

    cores = O.threads()
    per, macs, t = grow(target_s)
    # the same loops on one thread, on a smaller sample
    O.set_threads(1)
    try:
        per1, macs1, t1 = grow(target_s / 3)
    finally:
        O.set_threads(cores)
    return {"value": round(2.0 * macs / t / 1e12, 6), "unit": "TOP/s", "cores": cores, "kind": "oracle",
            "sample": sample(per, macs, t),
            "value_1_thread": round(2.0 * macs1 / t1 / 1e12, 6), "sample_1_thread": sample(per1, macs1, t1),
            "host_cpu": host_cpu(), "nproc": os.cpu_count()}


def host_cpu():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# ------------------------------------------------------------------ traffic from committed counters

def traffic_for(group, workload, layers):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary of this workload
    (profiles/traffic_<workload>.json, or profiles/traffic.json when it
    names the workload), if it was taken on the current kernel source and
    the group held the same layers there (else None)."""
    from paper_2006_10226_amd.rocprof_summary import kernel_source_sha1
    for name in (f"traffic_{workload}.json", "traffic.json"):
        path = os.path.join(ROOT, "profiles", name)
        if not os.path.exists(path):
            continue
        try:
            rec = json.load(open(path))
            if rec.get("workload") != workload or rec.get("source_sha1") != kernel_source_sha1(ROOT):
                return None
            g = rec.get("groups", {}).get(group, {})
            if sorted(g.get("layers", [])) != sorted(layers):
                return None
            return g.get("bytes_per_launch")
        except Exception:
            return None
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet50_b32")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the vendor int8 GEMM (torch._int_mm) on every layer's GEMM shape, warm, "
                         "as a reference point")
    ap.add_argument("--no-fuse", action="store_true",
                    help="chained workloads: run every residual add as its own kernel")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-warm-clock", action="store_true",
                    help="skip the warm per-layer timing and the clock reading (short counter runs)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (3 times), for scaling the "
                         "FETCH_SIZE / WRITE_SIZE counters, and exit")
    ap.add_argument("--layers-out", default=None, help="write per-layer timings as JSON to this file")
    ap.add_argument("--tuning-file", default=None,
                    help="kernel-choice file: reuse the choices recorded there, append newly timed ones "
                         "(default for the ResNet-50 b32 workload: a copy of the committed choices)")
    ap.add_argument("--retune", action="store_true",
                    help="time the candidate kernels on this machine instead of taking the committed choices")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {n} bytes 3 times")
        return
    choice = "timed on this machine"
    if args.tuning_file is None and not args.retune and args.workload in CHOICE_FILES:
        src = os.path.join(ROOT, CHOICE_FILES[args.workload])
        if os.path.exists(src):
            import shutil
            import tempfile
            fd, args.tuning_file = tempfile.mkstemp(prefix="qnn_choices_", suffix=".txt")
            os.close(fd)
            shutil.copyfile(src, args.tuning_file)   # a copy: newly timed shapes are appended to it, not to src
            choice = CHOICE_FILES[args.workload]
    elif args.tuning_file:
        choice = args.tuning_file
    if args.tuning_file:
        from paper_2006_10226_amd import qnn
        qnn.set_tuning_file(args.tuning_file)
    log(f"setting up {args.workload}")
    items, batch = setup(args.workload, fuse=not args.no_fuse)
    total_macs = sum(it.macs for it in items)
    total_bytes = sum(it.bytes for it in items)
    log(f"{len(items)} layers, {total_macs / 1e9:.2f} G MAC per step")

    ms, graph = time_steps(items, args.steps, args.warmup, not args.no_graph)
    graphed = graph is not None
    if graphed:
        # a graph replay has a fixed launch cost that dominates a step of
        # one or two small layers; such steps are timed as eager launches
        ms_eager, _ = time_steps(items, args.steps, args.warmup, False)
        log(f"step {ms:.4f} ms from a graph, {ms_eager:.4f} ms eager")
        if ms_eager < ms:
            ms, graphed = ms_eager, False
    value = 2.0 * total_macs / (ms * 1e-3) / 1e12
    log(f"step {ms:.4f} ms -> {value:.1f} TOP/s (graph={graphed})")

    per, how = time_launches(items, args.steps)
    if args.no_warm_clock:
        warm, clock = np.full(len(items), np.nan), None
    else:
        warm = time_warm(items)
        clock = sample_clock(items, graph if graphed else None)
        log(f"GPU clock while stepping: {clock}")
    lib_ms = library_gemm(items) if args.library_gemm else np.full(len(items), np.nan)
    groups = {}
    for it, t in zip(items, per):
        g = kernel_group(it)
        d = groups.setdefault(g, {"launches": 0, "ms": 0.0, "macs": 0, "bytes": 0, "layers": []})
        d["launches"] += 1
        d["ms"] += float(t)
        d["macs"] += it.macs
        d["bytes"] += it.bytes
        d["layers"].append(it.name)
    dom = max(groups, key=lambda g: groups[g]["ms"])
    D = groups[dom]
    # The dominant group's average kernel duration, from the events its main
    # kernels recorded at their own start and end (the duration rocprofv3's
    # kernel trace reports).  The step also holds the dispatch gaps between
    # kernels; the layers' shares of the step (for the aggregates below)
    # spread them in proportion to the kernel times.
    scale = ms / float(np.sum(per))
    avg_ms = D["ms"] / D["launches"]
    # the group's bound is the lower of its two roofs: a conv or dense group
    # whose algorithmic ops per byte sit above the ridge (peak ops / peak
    # bytes) is bound by the matrix cores, below it by HBM (as depthwise,
    # requantize and add always are)
    ridge = PEAK_INT8_TOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    mfma_bound = D["macs"] > 0 and dom.startswith("conv_") and 2.0 * D["macs"] / max(D["bytes"], 1) >= ridge
    if mfma_bound:
        achieved = 2.0 * D["macs"] / D["launches"] / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                "frac": round(achieved / PEAK_INT8_TOPS, 4)}
    else:
        achieved = D["bytes"] / D["launches"] / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["traffic"] = traffic_for(dom, args.workload, D["layers"])
    roof["kernel"] = dom
    roof["avg_launch_us"] = round(avg_ms * 1e3, 3)
    roof["avg_launch_us_step_share"] = round(avg_ms * scale * 1e3, 3)
    roof["launches_per_step"] = D["launches"]
    roof["layers"] = D["layers"]

    def roofline_us(it):
        return max(2.0 * it.macs / (PEAK_INT8_TOPS * 1e12), it.bytes / (PEAK_HBM_GBS * 1e9)) * 1e6

    roof_us = sum(roofline_us(it) for it in items)
    # Layers whose own roofline lets them reach at least 70% of the MFMA
    # peak (ops per byte at or above 0.7 x the ridge: the 3x3 convs and the
    # 1x1 convs with many input channels), aggregated over their share of
    # the step; the whole stack's ceiling beside it.
    cb = [(it, float(t) * scale) for it, t in zip(items, per)
          if it.macs and 2.0 * it.macs / max(it.bytes, 1) >= 0.7 * ridge]
    compute_bound = None
    if cb:
        cb_ops = sum(2.0 * it.macs for it, _ in cb)
        cb_ms = sum(t for _, t in cb)
        cb_roof_us = sum(roofline_us(it) for it, _ in cb)
        cb_tops = cb_ops / (cb_ms * 1e-3) / 1e12
        compute_bound = {"layers": len(cb), "tops": round(cb_tops, 1),
                         "frac_of_int8_peak": round(cb_tops / PEAK_INT8_TOPS, 4),
                         "ceiling_frac_of_int8_peak": round(cb_ops / (cb_roof_us * 1e-6) / 1e12 / PEAK_INT8_TOPS, 4),
                         "share_of_step": round(cb_ms / ms, 4)}
    layer_rows = []
    for it, t, h, tw, tl in zip(items, per, how, warm, lib_ms):
        row = {"layer": it.name, "kind": it.kind, "plan": it.desc, "us": round(float(t) * 1e3, 3), "timed": h,
               "warm_us": None if np.isnan(tw) else round(float(tw) * 1e3, 3),
               "library_gemm_us": None if np.isnan(tl) else round(float(tl) * 1e3, 3),
               "gmac": round(it.macs / 1e9, 4), "mbytes": round(it.bytes / 1e6, 3)}
        if it.macs:
            row["tops"] = round(2 * it.macs / (float(t) * 1e-3) / 1e12, 1)
        row["gbs"] = round(it.bytes / (float(t) * 1e-3) / 1e9, 1)
        row["roofline_us"] = round(roofline_us(it), 3)
        row["frac_of_roofline"] = round(roofline_us(it) / (float(t) * 1e3), 4)
        if it.macs:
            row["frac_of_int8_peak"] = round(row["tops"] / PEAK_INT8_TOPS, 4)
        layer_rows.append(row)
    if args.layers_out:
        os.makedirs(os.path.dirname(os.path.abspath(args.layers_out)), exist_ok=True)
        with open(args.layers_out, "w") as f:
            json.dump({"workload": args.workload, "step_ms": ms, "groups": groups, "layers": layer_rows}, f,
                      indent=1)
    for r in layer_rows:
        log(f"  {r['layer']:<24} {r['us']:9.2f} us  {r.get('tops', 0):8.1f} TOP/s {r['gbs']:8.1f} GB/s  {r['plan']}")

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(args.workload)
        log(f"cpu oracle: {cpu}")

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded, architecture shapes only, random weights)",
        "config": {"workload": args.workload, "batch": batch, "layers": len(items), "kernel_choice": choice,
                   "gmac_per_step": round(total_macs / 1e9, 3), "launch": "hipGraph" if graphed else "eager",
                   "frac_of_int8_peak": round(value / PEAK_INT8_TOPS, 4),
                   # sum over layers of max(MFMA time at peak, algorithmic bytes at HBM peak),
                   # over the measured step: the whole stack's fraction of its roofline
                   "stack_roofline_frac": round(roof_us / (ms * 1e3), 4),
                   # the best the stack could reach: every layer at its own roofline
                   "stack_ceiling_frac_of_int8_peak": round(2.0 * total_macs / (roof_us * 1e-6) / 1e12
                                                            / PEAK_INT8_TOPS, 4),
                   "compute_bound_layers": compute_bound,
                   # kernel times summed over the layers: cold (inside the step, each layer's
                   # inputs last touched a step earlier) and warm (each layer repeated back to back)
                   "layer_kernel_sum_us": {"cold": round(float(np.sum(per)) * 1e3, 2),
                                           "warm": None if args.no_warm_clock
                                           else round(float(np.sum(warm)) * 1e3, 2)},
                   "gpu_clock_mhz": clock,
                   # residual adds run inside the epilogue of a conv (chained workloads)
                   **({"fused_adds": sum(1 for it in items if getattr(it, "residual", None) is not None)}
                      if args.workload in CHAINS else {})},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    if args.library_gemm:
        gemm = [(float(tl), float(tw)) for tl, tw in zip(lib_ms, warm) if not np.isnan(tl)]
        out["library_gemm"] = {
            "what": "torch._int_mm (hipBLASLt) on each conv/dense layer's GEMM shape: int32 output, no gather, "
                    "zero-point terms or requantize; warm, back to back from a graph",
            "layers": len(gemm), "us_sum": round(sum(g for g, _ in gemm) * 1e3, 2),
            "this_library_warm_us_sum": None if args.no_warm_clock else round(sum(w for _, w in gemm) * 1e3, 2)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
