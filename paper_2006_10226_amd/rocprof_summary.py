"""Condense rocprofv3 CSV output of bench.py into short text summaries.

Reads
  * a ``--kernel-trace --stats --output-format csv`` directory (kernel_stats.csv),
  * two ``--pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` directories of the same
    bench command (counter_collection.csv, values in KiB per dispatch),
  * two more of ``bench.py --calibrate-copy MIB`` (a plain copy of known size),
  * the per-layer file bench.py writes (algorithmic bytes per kernel group),
and writes a markdown summary plus ``traffic.json``, which bench.py reads to
fill ``roofline.traffic`` as long as the kernel sources are unchanged.

and, when given, two more counter passes of the same bench command:
  * --mfma D: SQ_INSTS_VALU_MFMA_MOPS_I8 (int8 MFMA work in units of 512
    ops), SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE (MFMA busy fraction
    = busy cycles summed over the SIMDs / (traced kernel duration x 2.4 GHz
    x 1024 SIMDs); under counter collection GRBM_GUI_ACTIVE is stretched);
  * --l2 D: TCC_HIT_sum, TCC_MISS_sum (L2 hit rate), TCP_TCC_READ_REQ_sum
    and TCP_TCC_READ_REQ_LATENCY_sum (average L1-to-L2 read latency, cycles).

Usage:
  python -m paper_2006_10226_amd.rocprof_summary --stats D --fetch D --write D \
      --copy-fetch D --copy-write D --copy-mib 512 --layers F --out-md F \
      --out-json F [--mfma D] [--l2 D] --command "..." [--command "..."]
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import re

_CONV = re.compile(r"conv_mfma_kernel<(\d+), ?(\d+), ?(\d+), ?(\d+), ?(\d+), ?(\d+), ?(\d+)>")
_TAP = re.compile(r"conv_tap_kernel<(\d+), ?(\d+), ?(\d+), ?(\d+), ?(\d+)(?:, ?(true|false))?>")
_DMA = re.compile(r"conv_dma_kernel<(\d+), ?(\d+), ?(\d+), ?(\d+), ?(\d+), ?(true|false), ?(true|false)"
                  r"(?:, ?(\d+))?(?:, ?(true|false))?(?:, ?(true|false))?>")
_WAVE = re.compile(r"conv_wave_kernel<(\d+), ?(\d+), ?(true|false)>")
_HALO = re.compile(r"conv_halo_kernel<(\d+), ?(true|false)>")
_WIN = re.compile(r"conv_window_kernel<(\d+), ?(\d+), ?(\d+), ?(true|false)>")
# streaming window configurations (bands, reduction split, 16-channel blocks), in plan tile order
_WIN_CFGS = [(4, 2, 2), (2, 2, 2), (4, 1, 2), (8, 1, 2)]


def kernel_source_sha1(root=None):
    """SHA-1 over every kernel and library source (csrc/*), in name order:
    counters taken on other sources no longer describe the kernels."""
    if root is None:
        root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    h = hashlib.sha1()
    d = os.path.join(root, "paper_2006_10226_amd", "csrc")
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            h.update(open(os.path.join(d, name), "rb").read())
    return h.hexdigest()


def group_of(kernel_name):
    """bench.py's kernel-group name of a dispatched kernel symbol."""
    m = _CONV.search(kernel_name)
    if m:
        tc, tp, bk, _, _, avec, _ = (int(v) for v in m.groups())
        return f"conv_mfma tile={tc}x{tp}x{bk} gather={avec}"
    m = _TAP.search(kernel_name)
    if m:
        tc, tp, bk, wc, wp = (int(v) for v in m.groups()[:5])
        fused = " +add" if m.group(6) == "true" else ""
        return f"conv_tap tile={tc}x{tp}x{bk} threads={wc * wp * 64} stages=2{fused}"
    m = _DMA.search(kernel_name)
    if m:
        tc, tp, wc, wp, ns = (int(v) for v in m.groups()[:5])
        short = "s" if m.group(7) == "true" else ""
        ks = int(m.group(8)) if m.group(8) else 1
        split = " ksplit" if m.group(9) == "true" else ""
        fused = " +add" if m.group(10) == "true" else ""
        return f"conv_dma tile={tc}x{tp}x64 threads={wc * wp * ks * 64} stages={ns}{short}{split}{fused}"
    m = _WAVE.search(kernel_name)
    if m:
        split = int(m.group(1))
        return f"conv_wave tile=64x64x64 threads={max(4, split) * 64} stages={m.group(2)} split={split}"
    m = _HALO.search(kernel_name)
    if m:
        return f"conv_halo tile=64x64x64 threads={int(m.group(1)) * 64} stages=1"
    m = _WIN.search(kernel_name)
    if m:
        nb, ks, tcb = (int(v) for v in m.groups()[:3])
        cfg = _WIN_CFGS.index((nb, ks, tcb)) if (nb, ks, tcb) in _WIN_CFGS else -1
        return f"conv_window tile={16 * tcb}x64x64 threads={nb * ks * 64} stages=2 cfg={cfg}"
    base = kernel_name.split("(")[0].split("<")[0].replace("void ", "").strip()
    if base in ("qnn::depthwise3_kernel", "qnn::depthwise3_band_kernel", "qnn::depthwise_kernel"):
        return "depthwise"
    if base == "qnn::add_kernel":
        return "add"
    return base


def _one(pattern):
    files = glob.glob(pattern, recursive=True)
    if not files:
        raise SystemExit(f"no file matches {pattern}")
    return files[0]


def read_stats(d):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*kernel_stats.csv")))))
    out = []
    for r in rows:
        out.append({"name": r["Name"], "calls": int(r["Calls"]), "total_ns": float(r["TotalDurationNs"]),
                    "avg_ns": float(r["AverageNs"]), "pct": float(r["Percentage"]),
                    "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"])})
    return out


def read_counter(d, counter):
    """Per kernel group: list of per-dispatch counter values (summed over the
    counter's instances)."""
    return {g: [v[counter] for v in rows] for g, rows in read_counters(d, [counter]).items()}


def read_counters(d, counters):
    """Per kernel group: list of per-dispatch dicts {counter: value}, for the
    dispatches that report every one of `counters`."""
    vals = {}
    for r in csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))):
        if r["Counter_Name"] not in counters:
            continue
        key = (r["Dispatch_Id"], r["Kernel_Name"])
        row = vals.setdefault(key, {})
        row[r["Counter_Name"]] = row.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    per = {}
    for (_, name), row in vals.items():
        if all(c in row for c in counters):
            per.setdefault(group_of(name), []).append(row)
    return per


SIMDS = 256 * 4   # MI355X: 256 CUs of 4 SIMDs
CLOCK_HZ = 2.4e9  # MI355X peak engine clock


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--stats", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-fetch", required=True)
    ap.add_argument("--copy-write", required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--layers", required=True)
    ap.add_argument("--out-md", required=True)
    ap.add_argument("--out-json", required=True)
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--bench-json", help="the JSON line bench.py printed in the unprofiled run")
    ap.add_argument("--mfma", help="--pmc SQ_INSTS_VALU_MFMA_MOPS_I8 SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE directory")
    ap.add_argument("--l2", help="--pmc TCC_HIT_sum TCC_MISS_sum TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum "
                                 "directory")
    args = ap.parse_args()

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sha = kernel_source_sha1(root)

    stats = read_stats(args.stats)
    layers = json.load(open(args.layers))
    fetch = read_counter(args.fetch, "FETCH_SIZE")
    write = read_counter(args.write, "WRITE_SIZE")
    copy_bytes = args.copy_mib << 20
    cf = max(read_counter(args.copy_fetch, "FETCH_SIZE").values(), key=len)
    cw = max(read_counter(args.copy_write, "WRITE_SIZE").values(), key=len)
    # the copy's largest dispatches are the copy itself
    f_read = max(cf) * 1024.0 / copy_bytes
    f_write = max(cw) * 1024.0 / copy_bytes

    groups = {}
    for g, d in layers["groups"].items():
        if g not in fetch or g not in write:
            continue
        rd = sum(fetch[g]) / len(fetch[g]) * 1024.0 / f_read
        wr = sum(write[g]) / len(write[g]) * 1024.0 / f_write
        groups[g] = {"bytes_per_launch": round(rd + wr), "read_bytes_per_launch": round(rd),
                     "write_bytes_per_launch": round(wr),
                     "algorithmic_bytes_per_launch": round(d["bytes"] / d["launches"]),
                     "dispatches_counted": len(fetch[g]), "layers": sorted(d.get("layers", []))}
    # kernel time of each group from the trace (the duration bench.py's
    # roofline line must agree with)
    trace = {}
    for st in stats:
        gname = group_of(st["name"])
        t = trace.setdefault(gname, [0, 0.0])
        t[0] += st["calls"]
        t[1] += st["total_ns"]
    for g, d in layers["groups"].items():
        if g in groups and g in trace:
            groups[g]["trace_avg_us"] = round(trace[g][1] / trace[g][0] / 1e3, 3)
            groups[g]["algorithmic_ops_per_launch"] = round(2 * d["macs"] / d["launches"])
    if args.mfma:
        mf = read_counters(args.mfma, ["SQ_INSTS_VALU_MFMA_MOPS_I8", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"])
        for g, rows in mf.items():
            if g not in groups:
                continue
            n = len(rows)
            groups[g]["mfma_i8_ops_per_launch"] = round(sum(r["SQ_INSTS_VALU_MFMA_MOPS_I8"] for r in rows) / n * 512)
            busy = sum(r["SQ_VALU_MFMA_BUSY_CYCLES"] for r in rows) / n
            groups[g]["mfma_busy_cycles_per_launch"] = round(busy)
            # busy cycles summed over the SIMDs, over the kernel's traced
            # duration at the 2.4 GHz peak clock times 1024 SIMDs (the
            # counter passes themselves stretch GRBM_GUI_ACTIVE)
            t = groups[g].get("trace_avg_us")
            if t:
                groups[g]["mfma_busy"] = round(busy / (t * 1e-6 * CLOCK_HZ * SIMDS), 4)
    if args.l2:
        l2 = read_counters(args.l2, ["TCC_HIT_sum", "TCC_MISS_sum", "TCP_TCC_READ_REQ_sum",
                                     "TCP_TCC_READ_REQ_LATENCY_sum"])
        for g, rows in l2.items():
            if g not in groups:
                continue
            hit = sum(r["TCC_HIT_sum"] for r in rows)
            miss = sum(r["TCC_MISS_sum"] for r in rows)
            req = sum(r["TCP_TCC_READ_REQ_sum"] for r in rows)
            lat = sum(r["TCP_TCC_READ_REQ_LATENCY_sum"] for r in rows)
            groups[g]["l2_hit_rate"] = round(hit / max(1.0, hit + miss), 4)
            groups[g]["l1_to_l2_read_latency_cycles"] = round(lat / max(1.0, req), 1)
    rec = {"source_sha1": sha, "copy_mib": args.copy_mib, "fetch_scale": f_read, "write_scale": f_write,
           "workload": layers["workload"], "groups": groups}
    with open(args.out_json, "w") as f:
        json.dump(rec, f, indent=1)

    by_group = {}
    for s in stats:
        g = group_of(s["name"])
        d = by_group.setdefault(g, {"calls": 0, "total_ns": 0.0, "pct": 0.0})
        d["calls"] += s["calls"]
        d["total_ns"] += s["total_ns"]
        d["pct"] += s["pct"]
    lines = [f"# rocprofv3 summary: {layers['workload']}", ""]
    lines.append("Commands (run from the repository root of a copy of this tree):")
    lines.append("")
    for c in args.command:
        lines.append(f"    {c}")
    lines.append("")
    lines.append(f"kernel source digest (rocprof_summary.kernel_source_sha1) at the time: `{sha}`")
    lines.append("")
    if args.bench_json:
        lines.append("bench.py line of the unprofiled run:")
        lines.append("")
        lines.append("    " + open(args.bench_json).read().strip().splitlines()[-1])
        lines.append("")
    lines.append("## Kernel time (--kernel-trace --stats)")
    lines.append("")
    lines.append("| kernel group | calls | total ms | avg us | % |")
    lines.append("|---|---|---|---|---|")
    for g, d in sorted(by_group.items(), key=lambda kv: -kv[1]["total_ns"]):
        lines.append(f"| {g} | {d['calls']} | {d['total_ns'] / 1e6:.3f} | {d['total_ns'] / d['calls'] / 1e3:.3f} |"
                     f" {d['pct']:.1f} |")
    lines.append("")
    lines.append("## bench.py per-launch event timing of the same groups (unprofiled run)")
    lines.append("")
    lines.append("| kernel group | launches/step | avg us |")
    lines.append("|---|---|---|")
    for g, d in layers["groups"].items():
        lines.append(f"| {g} | {d['launches']} | {d['ms'] / d['launches'] * 1e3:.3f} |")
    lines.append("")
    lines.append("## HBM traffic (--pmc FETCH_SIZE, --pmc WRITE_SIZE)")
    lines.append("")
    lines.append(f"Copy calibration: a {args.copy_mib} MiB device copy read {max(cf):.0f} KiB and wrote "
                 f"{max(cw):.0f} KiB per dispatch, so counter KiB x 1024 / {f_read:.4f} (reads) and "
                 f"/ {f_write:.4f} (writes) give bytes.")
    lines.append("")
    lines.append("| kernel group | read MB/launch | write MB/launch | total MB/launch | algorithmic MB/launch |"
                 " ratio |")
    lines.append("|---|---|---|---|---|---|")
    for g, d in groups.items():
        lines.append(f"| {g} | {d['read_bytes_per_launch'] / 1e6:.3f} | {d['write_bytes_per_launch'] / 1e6:.3f} |"
                     f" {d['bytes_per_launch'] / 1e6:.3f} | {d['algorithmic_bytes_per_launch'] / 1e6:.3f} |"
                     f" {d['bytes_per_launch'] / max(1, d['algorithmic_bytes_per_launch']):.2f} |")
    lines.append("")
    if args.mfma or args.l2:
        lines.append("## Matrix cores and L2 (--pmc SQ_INSTS_VALU_MFMA_MOPS_I8 SQ_VALU_MFMA_BUSY_CYCLES "
                     "GRBM_GUI_ACTIVE; --pmc TCC_HIT_sum TCC_MISS_sum TCP_TCC_READ_REQ_sum "
                     "TCP_TCC_READ_REQ_LATENCY_sum)")
        lines.append("")
        lines.append("MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES (summed over the SIMDs; 16 per 16x16x64 int8 MFMA) / "
                     "(traced kernel duration x 2.4 GHz x 1024 SIMDs); int8 MFMA ops = "
                     "SQ_INSTS_VALU_MFMA_MOPS_I8 x 512, beside the algorithmic 2 x MACs (the difference is the "
                     "padding of the reduction and of partial tiles); L2 hit rate = TCC_HIT / (TCC_HIT + TCC_MISS); "
                     "L1-to-L2 read latency = TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ (cycles).")
        lines.append("")
        lines.append("| kernel group | layers | trace avg us | algorithmic GOP/launch | MFMA int8 GOP/launch |"
                     " MFMA busy | TOP/s (trace) | L2 hit rate | L1->L2 read latency (cycles) |")
        lines.append("|---|---|---|---|---|---|---|---|---|")
        for g, d in groups.items():
            ops = d.get("algorithmic_ops_per_launch", 0)
            t = d.get("trace_avg_us")
            tops = f"{ops / (t * 1e-6) / 1e12:.1f}" if t and ops else "-"
            mops = d.get("mfma_i8_ops_per_launch")
            lines.append(f"| {g} | {len(d['layers'])} | {t if t else '-'} | {ops / 1e9:.3f} |"
                         f" {mops / 1e9 if mops is not None else float('nan'):.3f} |"
                         f" {d.get('mfma_busy', float('nan')):.3f} | {tops} | {d.get('l2_hit_rate', float('nan')):.3f} |"
                         f" {d.get('l1_to_l2_read_latency_cycles', float('nan'))} |")
        lines.append("")
    lines.append("## Layers of each group")
    lines.append("")
    for g, d in groups.items():
        lines.append(f"- {g}: {', '.join(d['layers'])}")
    lines.append("")
    with open(args.out_md, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


if __name__ == "__main__":
    main()
