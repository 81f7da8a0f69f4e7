#!/usr/bin/env python3
"""Benchmark of the MI355X Kronecker-sparse matmul (Y = X K^T, K with support
I_a (x) 1_{b x c} (x) I_d) against the MI355X roofline.

Workload (the metric is the median over it): the pattern sweep
a in {1,2,4,8}, b, c in {16,32,48,64,96,128}, d in {1,2,4,8,16} with
a*b*d <= 8192 and a*c*d <= 8192 (700 patterns), batch B in {4096, 25088},
fp32 and bf16 (fp32 accumulate), batch-size-first and batch-size-last:
5600 points.  X and K are i.i.d. N(0, 1), synthetic.

Per point the fused method's minimum traffic (X read once, K read once, Y
written once; paper Section 4.3) and work are
    bytes = (B*N + B*M + a*b*c*d) * s,    flops = 2 * B * a*b*c*d,
the roof time is max(bytes / 8.0 TB/s, flops / peak) with peak = 157.3 TFLOP/s
(fp32) or 2516.6 TFLOP/s (bf16 MFMA), and the point's fraction of roofline is
roof time / measured time.

Timing: every point is timed over a rotation of buffer sets (one X and one Y
region of two 3 GB pools per call) such that >= 768 MB, three times the 256 MB
Infinity Cache, pass between two uses of the same buffers (at least 8 sets).
One pass launches one ks_matmul per set; the passes are captured into HIP
graphs of at most 512 calls, replayed --warmup times untimed and then --steps
times between two HIP events recorded on the replay stream.  The point's time
per call is the elapsed time / (steps * sets): back-to-back calls on one
stream, as the paper times its kernels (a loop of calls divided by its
length).  This time feeds `value`.  Each point is also timed call by call
(32 calls spread over the rotation, each between its own HIP event pair on
the launch stream): the median and interquartile range of those per-launch
times are reported per point, with the median fraction they give overall.
ms_per_step is the sum over the timed points of the time per call, i.e. the
time of one pass over the sweep (one step).

Reported per point (the JSON line's "points", fields in "points_fields"):
pattern, batch, dtype, layout, time per call, GB/s, TFLOP/s, fraction of
roofline, binding roof, per-launch median and quartiles.

The roofline object is computed for the dominant kernel instance (the one with
the largest share of one step): achieved = algorithmic bytes (or flops) of
all its timed calls / their total time, and avg_launch_us = that total time /
number of calls, which is what a profiler's per-kernel average duration
reports for the same command (the event time also holds the gaps between
launches inside the graph).

Also reported: the same measurements for the other workload families (tiny,
butterfly factors and 10-chain, Monarch factors and 2-chain, Transformer-MLP
layers) as context, and the fp64 CPU oracle timed on a bounded sample on the
host cores (cpu_baseline).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--sample S]
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "KS matmul achieved GB/s & TFLOP/s, fraction of roofline (median over patterns)"
HBM_BW = 8.0e12
PEAK = {"f32": 157.3e12, "bf16": 2516.6e12, "f16": 2516.6e12, "fp8": 5033.2e12}
ESIZE = {"f32": 4, "bf16": 2, "f16": 2, "fp8": 1}     # bytes per element of X and K
YSIZE = {"f32": 4, "bf16": 2, "f16": 2, "fp8": 2}     # bytes per element of Y (fp8 inputs give bf16 outputs)
POOL_BYTES = 3 << 30
ROTATE_BYTES = 768 << 20    # distinct buffer bytes between two uses of a buffer (3x the 256 MB MALL)
MIN_SETS = 8
GRAPH_LAUNCHES = 512
PER_LAUNCH_SAMPLES = 32     # calls timed one by one (own event pair each) per point


def sweep_patterns():
    pats = []
    for a in (1, 2, 4, 8):
        for b in (16, 32, 48, 64, 96, 128):
            for c in (16, 32, 48, 64, 96, 128):
                for d in (1, 2, 4, 8, 16):
                    if a * b * d <= 8192 and a * c * d <= 8192:
                        pats.append((a, b, c, d))
    return pats


def roof(pattern, batch, dtype):
    a, b, c, d = pattern
    nnz = a * b * c * d
    nbytes = (batch * a * c * d + nnz) * ESIZE[dtype] + batch * a * b * d * YSIZE[dtype]
    flops = 2.0 * batch * nnz
    t_hbm = nbytes / HBM_BW
    t_flop = flops / PEAK[dtype]
    return nbytes, flops, max(t_hbm, t_flop), ("hbm" if t_hbm >= t_flop else "mfma")


def plan_field(desc, key):
    return dict(kv.split("=", 1) for kv in desc.split())[key]


# Translation units that build each kernel family (csrc/ file name prefix of
# the .hip files; the .cpp files that plan its launches, which decide the
# tiles and which calls run it, count too, as does ks_host.cpp).
KERNEL_FAMILY_SOURCES = {
    "ks_dma_kernel": "ks_dma_", "ks_dma_bsl_kernel": "ks_dma_", "ks_direct_c_kernel": "ks_direct_", "ks_direct_kernel": "ks_direct_",
    "ks_staged_kernel": "ks_staged_", "ks_masked_kernel": "ks_masked_", "ks_fp8_kernel": "ks_fp8",
    "ks_valu_bsl_kernel": "ks_valu", "ks_valu_bsf_kernel": "ks_valu", "ks_generic_kernel": "ks_generic",
    "ks_chain_fused_kernel": "ks_chain_fused", "ks_chain_mfma_kernel": "ks_chain_mfma", "ks_chain_bfly_kernel": "ks_chain_bfly",
}
KERNEL_FAMILY_PLANNERS = {"ks_dma_": "ks_staged_plan.cpp", "ks_staged_": "ks_staged_plan.cpp",
                          "ks_direct_": "ks_direct_plan.cpp", "ks_masked_": "ks_direct_plan.cpp"}


def _include_closure(paths):
    """The files and every header they include with #include "..." (resolved
    in csrc/ or include/), transitively."""
    import re
    dirs = [os.path.join(ROOT, "paper_2405_15013_amd", "csrc"), os.path.join(ROOT, "include")]
    seen, todo = set(), list(paths)
    while todo:
        p = todo.pop()
        if p in seen:
            continue
        seen.add(p)
        with open(p) as fh:
            for m in re.finditer(r'^#include "([^"]+)"', fh.read(), re.M):
                for d in dirs:
                    q = os.path.normpath(os.path.join(d, m.group(1)))
                    if os.path.exists(q):
                        todo.append(q)
                        break
    return sorted(seen)


def kernel_sources_sha1(kernel=None):
    """Hash of the sources the kernels are built from (and their build
    script): a traffic record taken from profiler counters is used only while
    this hash is unchanged.  With `kernel` (an instance name), only that
    kernel family's translation units and the headers they include."""
    import hashlib
    h = hashlib.sha1()
    csrc = os.path.join(ROOT, "paper_2405_15013_amd", "csrc")
    if kernel is None:
        files = [os.path.join(csrc, f) for f in sorted(os.listdir(csrc))
                 if f.endswith((".h", ".hip", ".cpp")) and f != "ks_verify.hip"]
    else:
        prefix = KERNEL_FAMILY_SOURCES[kernel.split("<")[0]]
        files = _include_closure([os.path.join(csrc, f) for f in sorted(os.listdir(csrc))
                                  if f.startswith(prefix) and f.endswith(".hip")])
        files += [os.path.join(csrc, f) for f in sorted({KERNEL_FAMILY_PLANNERS.get(prefix, "ks_host.cpp"),
                                                          "ks_host.cpp"})]
    for p in files + [os.path.join(csrc, "..", "build.py")]:
        with open(p, "rb") as fh:
            h.update(os.path.basename(p).encode() + b"\0" + fh.read())
    return h.hexdigest()


TRAFFIC_TAG = "traffic-record: "


def traffic_record(kernel, sample_every):
    """HBM bytes per launch of `kernel` from a committed counter summary
    (profiles/*.md), or None when there is none for the current sources and
    the same sweep sample."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    try:
        sha = kernel_sources_sha1(kernel)
    except KeyError:
        return None
    for f in sorted(os.listdir(pdir)):
        if not f.endswith(".md"):
            continue
        with open(os.path.join(pdir, f)) as fh:
            for line in fh:
                if line.startswith(TRAFFIC_TAG):
                    rec = json.loads(line[len(TRAFFIC_TAG):])
                    if (rec.get("kernel") == kernel and rec.get("sources_sha1") == sha
                            and rec.get("sample_every") == sample_every):
                        return rec
    return None


def counter_per_dispatch(csv_path, counter, name_filter=None):
    """Per-dispatch totals of one counter from a rocprofv3 counter_collection
    CSV (rows of one dispatch are summed over the counter's instances), for
    the dispatches whose kernel name (spaces removed, lower case) contains
    `name_filter`."""
    import csv
    per = {}
    names = {}
    with open(csv_path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            if name_filter is not None and name_filter not in r["Kernel_Name"].replace(" ", "").lower():
                continue
            per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
            names[r["Kernel_Name"]] = names.get(r["Kernel_Name"], 0) + 1
    return per, names


def copy_calibration(nbytes=64 << 20, pairs=8, reps=20):
    """A plain device-to-device copy of `nbytes`, `reps` times over `pairs`
    buffer pairs: the profiler's FETCH_SIZE / WRITE_SIZE of these dispatches
    against the known nbytes give the counters' scale."""
    import torch
    src = [torch.ones(nbytes, dtype=torch.uint8, device="cuda:0") for _ in range(pairs)]
    dst = [torch.zeros(nbytes, dtype=torch.uint8, device="cuda:0") for _ in range(pairs)]
    torch.cuda.synchronize()
    for r in range(reps):
        dst[r % pairs].copy_(src[r % pairs])
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "dispatches": reps}), flush=True)


COPY_FLOOR_MB = (0.5, 1, 2, 4, 8, 16, 32, 64, 128, 256)


def copy_floor(run):
    """Time a plain device copy (torch copy_, read n bytes and write n bytes)
    with the sweep's own protocol (buffer rotation >= 768 MB, HIP graphs, time
    per call): the fraction of the HBM roof that moving the same bytes reaches
    under that protocol, per size (the per-launch cost included)."""
    import torch
    xs = run.pool_x.view(torch.float32)
    ys = run.pool_y.view(torch.float32)
    rows = []
    for mb in COPY_FLOOR_MB:
        n = (int(mb * 2**20) // 2 // 4 + 63) // 64 * 64  # elements per side: mb MB moved in total
        nb = n * 4
        sets = max(1, min(xs.numel(), ys.numel()) // n)

        def launch(r, h, n=n):
            ys[r * n:(r + 1) * n].copy_(xs[r * n:(r + 1) * n])

        t, _ = run.time_calls(2 * nb, sets, launch)
        rows.append({"bytes": 2 * nb, "us": t * 1e6, "frac": 2 * nb / HBM_BW / t})
    return rows


def copy_floor_frac(rows, nbytes):
    """The copy floor's fraction at `nbytes` moved (log-linear in bytes between
    the measured sizes, the largest size's rate beyond them)."""
    pts = sorted((r["bytes"], r["us"]) for r in rows)
    if nbytes >= pts[-1][0]:
        us = pts[-1][1] * nbytes / pts[-1][0]
    elif nbytes <= pts[0][0]:
        us = pts[0][1]
    else:
        for (b0, u0), (b1, u1) in zip(pts, pts[1:]):
            if b0 <= nbytes <= b1:
                w = math.log(nbytes / b0) / math.log(b1 / b0)
                us = u0 + w * (u1 - u0)
                break
    return nbytes / HBM_BW / (us * 1e-6)


def points_summary(points_jsonl, out_md, command_lines, floor_json=None, lowest=50):
    """Per-class tables of a bench run's per-point records: for every (dtype,
    layout, batch) a b x c matrix of the median fraction of roofline over the
    sweep patterns with that (b, c), the class median beside the copy floor's
    (same bytes, same protocol; when `floor_json` holds a --copy-floor run),
    and the `lowest` points with the smallest fraction."""
    import statistics
    pts = [json.loads(l) for l in open(points_jsonl) if l.strip()]
    sweep = set(sweep_patterns())
    pts = [p for p in pts if p.get("epilogue") is None and p["dtype"] in ("f32", "bf16")
           and p["batch"] in (4096, 25088) and "frac" in p and tuple(p["pattern"]) in sweep]
    seen, uniq = set(), []
    for p in pts:  # one record per sweep point (the families repeat some)
        key = (tuple(p["pattern"]), p["batch"], p["dtype"], p["layout"])
        if key not in seen:
            seen.add(key)
            uniq.append(p)
    pts = uniq
    floor = json.load(open(floor_json))["copy_floor"] if floor_json else None
    bs = sorted({p["pattern"][1] for p in pts})
    cs = sorted({p["pattern"][2] for p in pts})
    lines = ["# Sweep points by class: median fraction of roofline", "",
             "Command (from the repository root):", "", "```"] + command_lines + ["```", "",
             "%d sweep points.  Fraction = roof time / time per call (graph replay over a >= 768 MB "
             "rotation, the number that feeds the bench's value)." % len(pts), ""]
    if floor:
        lines += ["Copy floor (plain device copy of the same number of bytes, same protocol): "
                  + ", ".join("%.3g MB %.3f" % (r["bytes"] / 1e6, r["frac"]) for r in floor) + ".", ""]
    lines += ["| class | points | median fraction | median copy-floor fraction | median fraction / copy floor | median GB/s |",
              "|---|---:|---:|---:|---:|---:|"]
    classes = [(dt, lay, bt) for dt in ("f32", "bf16") for lay in ("bsf", "bsl") for bt in (4096, 25088)]
    for dt, lay, bt in classes:
        c = [p for p in pts if (p["dtype"], p["layout"], p["batch"]) == (dt, lay, bt)]
        if not c:
            continue
        cf = statistics.median(copy_floor_frac(floor, p["bytes"]) for p in c) if floor else float("nan")
        rel = statistics.median(p["frac"] / copy_floor_frac(floor, p["bytes"]) for p in c) if floor else float("nan")
        lines.append("| %s %s B=%d | %d | %.3f | %.3f | %.2f | %.0f |" % (
            dt, lay.upper(), bt, len(c), statistics.median(p["frac"] for p in c), cf, rel,
            statistics.median(p["gbps"] for p in c)))
    if floor:
        lines.append("| all | %d | %.3f | %.3f | %.2f | %.0f |" % (
            len(pts), statistics.median(p["frac"] for p in pts),
            statistics.median(copy_floor_frac(floor, p["bytes"]) for p in pts),
            statistics.median(p["frac"] / copy_floor_frac(floor, p["bytes"]) for p in pts),
            statistics.median(p["gbps"] for p in pts)))
    lines.append("")
    for dt, lay, bt in classes:
        c = [p for p in pts if (p["dtype"], p["layout"], p["batch"]) == (dt, lay, bt)]
        if not c:
            continue
        lines += ["%s %s B=%d: median fraction by b (rows) and c (columns)" % (dt, lay.upper(), bt), "",
                  "| b \\ c | " + " | ".join(str(x) for x in cs) + " |", "|---" * (len(cs) + 1) + "|"]
        for b in bs:
            cells = []
            for cc in cs:
                v = [p["frac"] for p in c if p["pattern"][1] == b and p["pattern"][2] == cc]
                cells.append("%.2f" % statistics.median(v) if v else "")
            lines.append("| %d | " % b + " | ".join(cells) + " |")
        lines.append("")
    low = sorted(pts, key=lambda p: p["frac"])[:lowest]
    lines += ["The %d points with the smallest fraction:" % lowest, "",
              "| pattern (a,b,c,d) | B | dtype | layout | us | GB/s | fraction | bound | kernel |",
              "|---|---:|---|---|---:|---:|---:|---|---|"]
    for p in low:
        lines.append("| %s | %d | %s | %s | %.2f | %.0f | %.3f | %s | `%s` |" % (
            tuple(p["pattern"]), p["batch"], p["dtype"], p["layout"].upper(), p["us"], p["gbps"], p["frac"],
            p["bound"], p["kernel"]))
    lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


MFMA_COUNTERS = ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_WAIT_INST_ANY", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_MFMA",
                 "GRBM_GUI_ACTIVE")


def mfma_summary(csv_paths, out_md, command_lines):
    """MFMA utilisation of kernel instances from one counter pass each
    (rocprofv3 --pmc with MFMA_COUNTERS over `bench.py --kernel NAME --eager`):
    counters summed over the instance's dispatches, kernel time from their
    start and end timestamps, matrix-pipe busy fraction over the chip's 1024
    SIMDs at 2.4 GHz, and the fraction of wavefront cycles spent waiting."""
    import csv
    cols = []
    for path in csv_paths:
        tot, spans, kname = {}, {}, None
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if not r["Kernel_Name"].replace(" ", "").replace("void", "").startswith("ks::"):
                    continue
                kname = r["Kernel_Name"].replace("void ", "").replace(" ", "").split("(")[0]
                tot[r["Counter_Name"]] = tot.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                spans[r["Dispatch_Id"]] = (int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
        t = sum(e - b for b, e in spans.values()) * 1e-9
        busy = tot.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        cols.append({"kernel": kname, "dispatches": len(spans), "time_s": t, "mfma": tot.get("SQ_INSTS_MFMA", 0.0),
                     "busy": busy, "busy_frac": busy / (1024 * t * 2.4e9) if t else float("nan"),
                     "wait_frac": tot.get("SQ_WAIT_INST_ANY", 0.0) / max(1.0, tot.get("SQ_WAVE_CYCLES", 0.0)),
                     "waves": tot.get("SQ_WAVES", 0.0)})
    lines = ["# MFMA utilisation of the fp32 MFMA-bound instances over their sweep points", "",
             "Command (one counter pass per instance, from the repository root; the sweep points of the instance "
             "launched call by call):", "", "```"] + command_lines + ["```", "",
             "| | " + " | ".join("`%s`" % c["kernel"] for c in cols) + " |", "|---" + "|---:" * len(cols) + "|",
             "| dispatches | " + " | ".join("%d" % c["dispatches"] for c in cols) + " |",
             "| kernel time (sum) | " + " | ".join("%.2f ms" % (c["time_s"] * 1e3) for c in cols) + " |",
             "| SQ_INSTS_MFMA | " + " | ".join("%.4g" % c["mfma"] for c in cols) + " |",
             "| SQ_VALU_MFMA_BUSY_CYCLES | " + " | ".join("%.4g" % c["busy"] for c in cols) + " |",
             "| busy cycles per MFMA | " + " | ".join("%.1f" % (c["busy"] / max(1.0, c["mfma"])) for c in cols) + " |",
             "| MFMA busy / (1024 SIMDs x kernel time x 2.4 GHz) | " + " | ".join(
                 "%.2f" % c["busy_frac"] for c in cols) + " |",
             "| SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES | " + " | ".join("%.2f" % c["wait_frac"] for c in cols) + " |",
             "| SQ_WAVES | " + " | ".join("%.4g" % c["waves"] for c in cols) + " |", "",
             "Reading: the fp32 matrix pipes are busy %.0f-%.0f %% of these kernels' time (one 16x16x4 fp32 MFMA "
             "keeps a pipe busy 32 cycles) while the resident wavefronts wait on outstanding operations %.0f-%.0f %% "
             "of their cycles: these points are bound by latency inside the kernel, not by MFMA throughput." % (
                 100 * min(c["busy_frac"] for c in cols), 100 * max(c["busy_frac"] for c in cols),
                 100 * min(c["wait_frac"] for c in cols), 100 * max(c["wait_frac"] for c in cols)), ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


BUTTERFLY10 = [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]
MONARCH2 = [(1, 32, 32, 32), (32, 32, 32, 1)]


def chain_workloads(run):
    """The chain workloads, each as planned (fused where the planner fuses
    it) and factor by factor: the butterfly 10-chain (N = 1024) at batch
    4096 and the Monarch 2-chain (N = 1024) at batch 16384, fp32 and bf16,
    both layouts."""
    out = []
    for dtype in ("f32", "bf16"):
        run.fill(dtype)
        for pats, batch in ((BUTTERFLY10, 4096), (MONARCH2, 16384)):
            for layout in ("bsl", "bsf"):
                for fused in (True, False):
                    out.append(run.chain(pats, batch, dtype, layout, fused=fused))
    return out


def chain_summary(stats_csv, chains_jsonl, out_md, command_lines):
    """Write the chain workloads' timings (per call through HIP graphs, and
    the per-launch median) beside the device time rocprofv3 reports for each
    chain kernel of the same run."""
    import csv
    recs = [json.loads(l) for l in open(chains_jsonl) if l.strip()]
    rows = [r for r in csv.DictReader(open(stats_csv)) if "ks_chain_" in r["Name"]]
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# Chain workloads: fused kernels and factor by factor", "",
             "Butterfly 10-chain (2^(l-1), 2, 2, 2^(10-l)), l = 1..10, at batch 4096 and Monarch 2-chain "
             "(1,32,32,32)·(32,32,32,1) at batch 16384 (both N = 1024), fp32 and bf16, both layouts; each as "
             "planned and factor by factor; %s." % (
                 "per call: graph replay over a >= 768 MB buffer rotation; per launch: median of HIP events"), "",
             "Command (from the repository root):", "", "```"] + command_lines + ["```", "",
             "| chain | B | dtype | layout | path | us per call | us per launch (median) | fused bound us "
             "(X + ΣK + Y at 8 TB/s) | fraction of fused bound |",
             "|---|---:|---|---|---|---:|---:|---:|---:|"]
    for r in recs:
        lines.append("| %s | %d | %s | %s | %s | %.2f | %.2f | %.2f | %.3f |" % (
            "butterfly 10" if len(r["chain"]) == 10 else "Monarch 2", r["batch"], r["dtype"], r["layout"].upper(),
            r["path"], r["us"], r.get("launch_us_median", float("nan")), r["fused_lower_bound_us"],
            r["frac_fused_bound"]))
    lines += ["", "Device time of the chain kernels (rocprofv3, all dispatches of the run, warmup included):", "",
              "| kernel | calls | avg us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "")
        lines.append("| `%s` | %s | %.2f | %.2f | %.2f |" % (
            name, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def trace_summary(stats_csv, bench_json, out_md, command_lines, top=25):
    """Write the kernel-trace summary (rocprofv3 --kernel-trace --stats) of a
    bench run, with the dominant kernel's profiler average beside the
    bench's own avg_launch_us.  `bench_json` is the bench line of the same
    command run without the profiler (the tracer adds a per-dispatch cost
    that changes which instance dominates among microsecond-sized calls)."""
    import csv
    with open(bench_json) as fh:
        bench = json.loads(fh.read().strip().splitlines()[-1])
    dom = bench["roofline"]["kernel"]
    rows = list(csv.DictReader(open(stats_csv)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    drow = [r for r in rows if dom in r["Name"].replace(" ", "")]
    lines = ["# Kernel-trace summary: KS pattern sweep bench (all kernels)", "",
             "Workload: %s, %d timed sweep points plus the context families; %d timed + %d warmup passes per point "
             "over a >= 768 MB buffer rotation, launched through HIP graphs." % (
                 bench["config"]["workload"], bench["config"]["points"], bench["steps"], bench["warmup"]), "",
             "Command (from the repository root):", "", "```"] + command_lines + ["```", "",
             "Bench line of the same command without the profiler: median fraction of roofline %.4f "
             "(sources sha1 %s)." % (
                 bench["value"], bench["sources_sha1"][:12]), "",
             "Dominant kernel (largest share of timed sweep time, %.1f %%): `%s`." % (
                 100 * bench["roofline"].get("share_of_step_time", bench["roofline"].get("share_of_sweep_time", 0)), dom)]
    if drow:
        r = drow[0]
        lines.append("bench.py (HIP events on the replay stream, timed calls only): avg_launch_us = %.2f; "
                     "rocprofv3 average over all its dispatches: %.2f us (%s calls, incl. warmup and eager calls)." % (
                         bench["roofline"]["avg_launch_us"], float(r["AverageNs"]) / 1e3, r["Calls"]))
    lines += ["", "| Kernel | Calls | Total ms | Avg us | % |", "|---|---:|---:|---:|---:|"]
    for r in rows[:top]:
        name = r["Name"].replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0]
        lines.append("| `%s` | %s | %.1f | %.2f | %.2f |" % (name, r["Calls"], float(r["TotalDurationNs"]) / 1e6,
                                                          float(r["AverageNs"]) / 1e3, float(r["Percentage"])))
    lines.append("")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


def pmc_summary(pdir, out_md, command_lines):
    """Write the traffic summary of the dominant kernel from four counter
    passes in `pdir` (fetch.csv, write.csv: the kernel's sweep points;
    copy_fetch.csv, copy_write.csv: the copy calibration) and the bench line
    of the kernel's points (bench.json)."""
    with open(os.path.join(pdir, "bench.json")) as fh:
        bench = json.loads(fh.read().strip().splitlines()[-1])
    kernel = bench["roofline"]["kernel"]
    cal_bytes = 64 << 20
    # The copy's dispatches only (the buffers' fill kernels run in the same pass).
    cf, cfn = counter_per_dispatch(os.path.join(pdir, "copy_fetch.csv"), "FETCH_SIZE", "copy")
    cw, cwn = counter_per_dispatch(os.path.join(pdir, "copy_write.csv"), "WRITE_SIZE", "copy")
    import numpy as np
    f_cal = float(np.median(list(cf.values()))) * 1024.0
    w_cal = float(np.median(list(cw.values()))) * 1024.0
    f_scale, w_scale = cal_bytes / f_cal, cal_bytes / w_cal
    kf, kfn = counter_per_dispatch(os.path.join(pdir, "fetch.csv"), "FETCH_SIZE", kernel.lower())
    kw, kwn = counter_per_dispatch(os.path.join(pdir, "write.csv"), "WRITE_SIZE", kernel.lower())
    fetch = float(np.mean(list(kf.values()))) * 1024.0 * f_scale
    write = float(np.mean(list(kw.values()))) * 1024.0 * w_scale
    alg = bench["roofline"]["algorithmic_bytes_per_launch"]
    rec = {"kernel": kernel, "sources_sha1": kernel_sources_sha1(kernel), "sample_every": bench["config"]["sample_every"],
           "dispatches": [len(kf), len(kw)], "timed_calls": bench["roofline"]["timed_calls"],
           "fetch_scale": f_scale, "write_scale": w_scale,
           "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
           "traffic_bytes_per_launch": fetch + write, "algorithmic_bytes_per_launch": alg}
    lines = ["# HBM traffic of %s over its sweep points" % kernel, "",
             "Counter passes (rocprofv3 --pmc, one counter per run), each command run from the repository root:", "",
             "```"] + command_lines + ["```", "",
             "| | value |", "|---|---|",
             "| copy calibration kernel | %s |" % ", ".join(sorted(cfn)),
             "| copy of 64 MiB: FETCH_SIZE (median per dispatch) | %.1f MiB -> scale x%.3f |" % (f_cal / 2**20, f_scale),
             "| copy of 64 MiB: WRITE_SIZE (median per dispatch) | %.1f MiB -> scale x%.3f |" % (w_cal / 2**20, w_scale),
             "| kernel dispatches counted (fetch, write) | %d, %d |" % (len(kf), len(kw)),
             "| sweep points of the kernel | %d |" % bench["roofline"]["points"],
             "| algorithmic bytes per launch (X + K + Y once) | %.4g |" % alg,
             "| fetched bytes per launch (scaled) | %.4g (%.3f of the algorithmic bytes) |" % (fetch, fetch / max(1.0, alg)),
             "| written bytes per launch (scaled) | %.4g |" % write,
             "| HBM traffic per launch | %.4g (%.3f x algorithmic) |" % (fetch + write, (fetch + write) / max(1.0, alg)),
             "", TRAFFIC_TAG + json.dumps(rec), ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


class Runner:
    def __init__(self, steps, warmup, eager=False, per_launch=True):
        import torch
        import paper_2405_15013_amd as ks
        if not os.path.exists(ks.library_path()):
            from paper_2405_15013_amd import build
            build.build()
        self.torch = torch
        self.ks = ks
        self.lib = ks.load_library()
        self.steps = steps
        self.warmup = warmup
        self.dev = torch.device("cuda:0")
        self.pool_x = torch.empty(POOL_BYTES, dtype=torch.uint8, device=self.dev)
        self.pool_y = torch.empty(POOL_BYTES, dtype=torch.uint8, device=self.dev)
        self.stream = torch.cuda.Stream(device=self.dev)
        self.filled = None
        self.eager = eager
        self.per_launch = per_launch

    def fill(self, dtype):
        """Fill the input pool with N(0,1) values of the storage dtype."""
        torch = self.torch
        if self.filled == dtype:
            return
        g = torch.Generator(device=self.dev)
        g.manual_seed(20240523)
        chunk = 1 << 26
        if dtype == "fp8":  # N(0,1) drawn in bf16, rounded to E4M3
            view = self.pool_x.view(torch.float8_e4m3fn)
            for s in range(0, view.numel(), chunk):
                n = min(chunk, view.numel() - s)
                view[s:s + n] = torch.randn(n, device=self.dev, generator=g, dtype=torch.bfloat16).to(
                    torch.float8_e4m3fn)
        else:
            tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
            view = self.pool_x.view(tdt)
            for s in range(0, view.numel(), chunk):
                view[s:s + chunk].normal_(generator=g)
        torch.cuda.synchronize()
        self.filled = dtype

    def time_calls(self, set_bytes, nsets_pool, launch):
        """Time one call per buffer set over a rotation of >= ROTATE_BYTES.

        Every buffer set (one X and one Y region of the pools) is used once per
        pass, so at least ROTATE_BYTES of distinct memory pass between two uses
        of the same buffers.  The launches of a pass are captured into HIP
        graphs of at most GRAPH_LAUNCHES calls; `warmup` untimed passes are
        followed by `steps` timed passes, bracketed by HIP events recorded on
        the replay stream (the stream the kernels run on).
        `launch(r, stream_handle)` issues the call on buffer set r.
        Returns (seconds per call, calls per pass)."""
        torch = self.torch
        nsets = max(MIN_SETS, math.ceil(ROTATE_BYTES / max(1, set_bytes)))
        nsets = min(nsets, nsets_pool)
        if self.eager:
            return self.time_eager(nsets, launch), nsets
        graphs = []
        with torch.cuda.stream(self.stream):
            launch(0, self.stream.cuda_stream)  # eager call: plan creation outside the capture
            torch.cuda.synchronize()
            for g0 in range(0, nsets, GRAPH_LAUNCHES):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=self.stream):
                    hc = torch.cuda.current_stream().cuda_stream
                    for r in range(g0, min(nsets, g0 + GRAPH_LAUNCHES)):
                        launch(r, hc)
                graphs.append(g)
            for _ in range(self.warmup):
                for g in graphs:
                    g.replay()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            self.stream.synchronize()
            e0.record(self.stream)
            for _ in range(self.steps):
                for g in graphs:
                    g.replay()
            e1.record(self.stream)
            e1.synchronize()
        ms = e0.elapsed_time(e1)
        del graphs
        return ms * 1e-3 / (self.steps * nsets), nsets

    def time_per_launch(self, nsets, launch, count=PER_LAUNCH_SAMPLES):
        """Per-launch durations: `count` calls on buffer sets spread over the
        rotation, each between its own pair of HIP events on the launch stream
        (launched one by one, after a warm-up call on each set).  Returns
        (median, first quartile, third quartile) in seconds."""
        import numpy as np
        torch = self.torch
        sets = sorted(set(int(round(i * (nsets - 1) / max(1, count - 1))) for i in range(min(count, nsets))))
        with torch.cuda.stream(self.stream):
            h = self.stream.cuda_stream
            for r in sets:
                launch(r, h)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in sets]
            self.stream.synchronize()
            for (e0, e1), r in zip(ev, sets):
                e0.record(self.stream)
                launch(r, h)
                e1.record(self.stream)
            self.stream.synchronize()
        t = np.array([e0.elapsed_time(e1) * 1e-3 for e0, e1 in ev])
        return float(np.median(t)), float(np.quantile(t, 0.25)), float(np.quantile(t, 0.75))

    def time_eager(self, nsets, launch):
        """The same rotation launched call by call (no graphs), for profiler
        counter passes, which count per dispatch."""
        torch = self.torch
        with torch.cuda.stream(self.stream):
            h = self.stream.cuda_stream
            for _ in range(self.warmup):
                for r in range(nsets):
                    launch(r, h)
            self.stream.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            for _ in range(self.steps):
                for r in range(nsets):
                    launch(r, h)
            e1.record(self.stream)
            e1.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / (self.steps * nsets)

    def point(self, pattern, batch, dtype, layout, only_kernel=None, epilogue=False):
        torch = self.torch
        a, b, c, d = pattern
        s = ESIZE[dtype]
        N, M = a * c * d, a * b * d
        xb = (batch * N * s + 255) // 256 * 256
        yb = (batch * M * YSIZE[dtype] + 255) // 256 * 256
        tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16,
               "fp8": torch.float8_e4m3fn}[dtype]
        kv = torch.randn(a * d * b * c, device=self.dev).to(tdt)
        px, py = self.pool_x.data_ptr(), self.pool_y.data_ptr()
        lay = 0 if layout == "bsf" else 1
        dt = {"f32": 0, "bf16": 1, "f16": 2, "fp8": 3}[dtype]
        kp = kv.data_ptr()
        nsets_pool = max(1, POOL_BYTES // max(xb, yb))
        lib = self.lib

        bias = torch.randn(M, device=self.dev).to(torch.bfloat16 if dtype == "fp8" else tdt) if epilogue else None

        def launch(r, h):
            if epilogue:  # Y = GELU(X K^T + bias)
                st = lib.ks_matmul_bias_act(a, b, c, d, kp, bias.data_ptr(), 1, px + r * xb, py + r * yb, batch,
                                            lay, dt, h)
            else:
                st = lib.ks_matmul(a, b, c, d, kp, px + r * xb, py + r * yb, batch, lay, dt, h)
            if st != 0:
                raise RuntimeError("ks_matmul failed: %s" % self.ks.ks_status_string(st))

        try:
            desc0 = self.ks.ks_plan_describe(a, b, c, d, batch, layout, dtype)
        except self.ks.KsError:
            return None  # the forced variant cannot run this point
        if only_kernel is not None and plan_field(desc0, "kernel") != only_kernel:
            return None
        t, nsets = self.time_calls(xb + yb, nsets_pool, launch)
        nbytes, flops, t_roof, bound = roof(pattern, batch, dtype)
        desc = self.ks.ks_plan_describe(a, b, c, d, batch, layout, dtype)
        r = {"pattern": list(pattern), "batch": batch, "dtype": dtype, "layout": layout, "us": t * 1e6,
             "epilogue": "bias+gelu" if epilogue else None,
             "gbps": nbytes / t / 1e9, "tflops": flops / t / 1e12, "frac": t_roof / t, "bound": bound,
             "roof_us": t_roof * 1e6, "bytes": nbytes, "flops": flops, "calls_per_pass": nsets,
             "kernel": plan_field(desc, "kernel"), "plan": desc}
        if self.per_launch and not self.eager:
            med, q1, q3 = self.time_per_launch(nsets, launch)
            r.update({"launch_us_median": med * 1e6, "launch_us_iqr": [q1 * 1e6, q3 * 1e6],
                      "frac_launch_median": t_roof / med})
        return r

    def chain(self, patterns, batch, dtype, layout, fused=True):
        torch = self.torch
        ks = self.ks
        ks.ks_force_chain_fusion(None if fused else 0)
        try:
            return self._chain(patterns, batch, dtype, layout)
        finally:
            ks.ks_force_chain_fusion(None)

    def _chain(self, patterns, batch, dtype, layout):
        torch = self.torch
        ks = self.ks
        s = ESIZE[dtype]
        tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
        kvs = [torch.randn(p[0] * p[1] * p[2] * p[3], device=self.dev).to(tdt) for p in patterns]
        factors = [(p, k) for p, k in zip(patterns, kvs)]
        aL, bL, cL, dL = patterns[-1]
        a1, b1, c1, d1 = patterns[0]
        N, M = aL * cL * dL, a1 * b1 * d1
        xb = (batch * N * s + 255) // 256 * 256
        yb = (batch * M * s + 255) // 256 * 256
        wsb = ks.ks_chain_workspace_bytes(factors, batch, dtype)
        ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=self.dev)
        px, py = self.pool_x.data_ptr(), self.pool_y.data_ptr()
        nsets_pool = max(1, POOL_BYTES // max(xb, yb))

        def launch(r, h):
            ks.ks_chain(factors, px + r * xb, py + r * yb, batch, layout, dtype, ws, wsb, stream=h)

        t, nsets = self.time_calls(xb + yb, nsets_pool, launch)
        unfused = sum(roof(p, batch, dtype)[0] for p in patterns)
        fused = (batch * (N + M) + sum(p[0] * p[1] * p[2] * p[3] for p in patterns)) * s
        flops = sum(roof(p, batch, dtype)[1] for p in patterns)
        t_roof = max(unfused / HBM_BW, flops / PEAK[dtype])
        t_fused = max(fused / HBM_BW, flops / PEAK[dtype])
        desc = ks.ks_chain_describe(factors, batch, layout, dtype)
        r = {"chain": [list(p) for p in patterns], "batch": batch, "dtype": dtype, "layout": layout,
             "path": desc.split()[0], "us": t * 1e6, "gbps_unfused": unfused / t / 1e9, "frac_unfused": t_roof / t,
             "fused_lower_bound_us": t_fused * 1e6, "frac_fused_bound": t_fused / t,
             "gbps_fused_bytes": fused / t / 1e9}
        if self.per_launch:
            med, q1, q3 = self.time_per_launch(nsets, launch)
            r.update({"launch_us_median": med * 1e6, "launch_us_iqr": [q1 * 1e6, q3 * 1e6]})
        return r


def cpu_baseline(every_4096=14, every_25088=88):
    """The fp64 oracle timed on the host cores, on a bounded sample of the
    sweep: every `every_4096`-th pattern (50 of the 700) at batch 4096 and
    every `every_25088`-th (8) at batch 25088, both layouts.  The oracle does
    the same fp64 work whatever the storage type of its inputs, so each
    timed call is scored against both the fp32 and the bf16 roofline of its
    point.  Reported in the metric's unit (median fraction of the MI355X
    roofline over the sampled points) and in GB/s of algorithmic traffic.
    Inputs are N(0,1) values (numpy's default generator; only the oracle call
    is timed)."""
    import numpy as np
    import oracle
    fracs, gbps = [], []
    total = 0.0
    npts = {}
    rng = np.random.default_rng(20240523)
    for batch, every in ((4096, every_4096), (25088, every_25088)):
        pats = sweep_patterns()[::every]
        npts[batch] = len(pats)
        for p in pats:
            a, b, c, d = p
            x = rng.standard_normal((batch, a * c * d), dtype=np.float32).astype(np.float64)
            kv = rng.standard_normal(a * d * b * c, dtype=np.float32).astype(np.float64)
            for layout in ("bsf", "bsl"):
                xl = x if layout == "bsf" else np.ascontiguousarray(x.T)
                t0 = time.perf_counter()
                oracle.matmul(p, kv, xl, batch, layout)
                t = time.perf_counter() - t0
                total += t
                for dtype in ("f32", "bf16"):
                    nbytes, flops, t_roof, _ = roof(p, batch, dtype)
                    fracs.append(t_roof / t)
                    gbps.append(nbytes / t / 1e9)
            del x
    return {"value": float(np.median(fracs)), "unit": "fraction of MI355X roofline (median over sampled points)",
            "gbps_median": float(np.median(gbps)), "cores": oracle.threads(), "kind": "oracle",
            "seconds": total,
            "sample": "%d sweep patterns at batch 4096 (every %dth) and %d at batch 25088 (every %dth), BSF and BSL, "
                      "each timed call scored against its fp32 and its bf16 point: %d points, fp64 arithmetic"
                      % (npts[4096], every_4096, npts[25088], every_25088, len(fracs))}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--sample", type=int, default=1,
                    help="time a seeded 1/S subset of the sweep points (1 = all 5600)")
    ap.add_argument("--points-out", default=None,
                    help="also write every timed point as one JSON line to this file")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-families", action="store_true")
    ap.add_argument("--variant", type=int, default=-1,
                    help="force a kernel variant for the sweep points (tuning; points it cannot run are skipped)")
    ap.add_argument("--kernel", default=None,
                    help="time only the sweep points whose plan runs this kernel instance (counter passes)")
    ap.add_argument("--eager", action="store_true", help="launch call by call instead of through HIP graphs")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the plain 64 MiB copy used to scale the profiler's byte counters")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("DIR", "OUT_MD"),
                    help="summarise counter passes in DIR into OUT_MD (no GPU)")
    ap.add_argument("--trace-summary", nargs=3, metavar=("STATS_CSV", "BENCH_JSON", "OUT_MD"),
                    help="summarise a rocprofv3 kernel_stats.csv of a bench run into OUT_MD (no GPU)")
    ap.add_argument("--copy-floor", default=None, metavar="OUT_JSON",
                    help="only time a plain device copy at 0.5-256 MB with the sweep's protocol, into OUT_JSON")
    ap.add_argument("--points-summary", nargs=2, metavar=("POINTS_JSONL", "OUT_MD"),
                    help="summarise a --points-out file by class into OUT_MD (no GPU)")
    ap.add_argument("--mfma-summary", nargs="+", metavar="CSV_THEN_OUT_MD",
                    help="summarise MFMA counter passes (counter_collection.csv files, then OUT_MD; no GPU)")
    ap.add_argument("--copy-floor-in", default=None, metavar="FLOOR_JSON",
                    help="a --copy-floor result for --points-summary")
    ap.add_argument("--chains", default=None, metavar="OUT_JSONL",
                    help="time only the chain workloads (butterfly 10-chain at batch 4096, Monarch 2-chain at "
                         "batch 16384; fp32 and bf16, both layouts, as planned and factor by factor) into OUT_JSONL")
    ap.add_argument("--chain-summary", nargs=3, metavar=("STATS_CSV", "CHAINS_JSONL", "OUT_MD"),
                    help="summarise a --chains run under rocprofv3 --kernel-trace --stats (no GPU)")
    ap.add_argument("--pmc-command", action="append", default=[],
                    help="command line recorded in the --pmc-summary / --trace-summary output (repeatable)")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.pmc_command)
        return
    if args.trace_summary:
        trace_summary(*args.trace_summary, args.pmc_command)
        return
    if args.mfma_summary:
        mfma_summary(args.mfma_summary[:-1], args.mfma_summary[-1], args.pmc_command)
        return
    if args.points_summary:
        points_summary(args.points_summary[0], args.points_summary[1], args.pmc_command, args.copy_floor_in)
        return
    if args.chain_summary:
        chain_summary(*args.chain_summary, args.pmc_command)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the KS matmul path shards over the batch with no "
              "communication, so there is no multi-GPU step to time (got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        copy_calibration()
        return
    if args.copy_floor:
        rows = copy_floor(Runner(args.steps, args.warmup, per_launch=False))
        with open(args.copy_floor, "w") as fh:
            json.dump({"copy_floor": rows}, fh)
        print(json.dumps({"copy_floor": rows}), flush=True)
        return
    if args.chains:
        run = Runner(args.steps, args.warmup)
        with open(args.chains, "w") as fout:
            for r in chain_workloads(run):
                fout.write(json.dumps(r) + "\n")
                print("[bench] chain %s B=%d %s %s %s: %.2f us" % (
                    "butterfly10" if len(r["chain"]) == 10 else "monarch2", r["batch"], r["dtype"], r["layout"],
                    r["path"], r["us"]), file=sys.stderr, flush=True)
        return
    t_start = time.time()
    run = Runner(args.steps, args.warmup, eager=args.eager)
    if args.points_out:
        os.makedirs(os.path.dirname(args.points_out) or ".", exist_ok=True)
    pats = sweep_patterns()
    grid = [(dtype, batch, layout, p) for dtype in ("f32", "bf16") for batch in (4096, 25088)
            for layout in ("bsf", "bsl") for p in pats]
    keep = np.random.default_rng(7).permutation(len(grid))[::args.sample]
    keep = set(int(k) for k in keep)
    points = []
    skipped = 0
    with open(args.points_out or os.devnull, "w") as fout:
        run.ks.ks_force_variant(args.variant if args.variant >= 0 else None)
        for idx, (dtype, batch, layout, p) in enumerate(grid):
            if idx not in keep:
                continue
            run.fill(dtype)
            r = run.point(p, batch, dtype, layout, only_kernel=args.kernel)
            if r is None:
                skipped += 1
                continue
            points.append(r)
            fout.write(json.dumps(r) + "\n")
            if len(points) % 200 == 0:
                print("[bench] %d/%d sweep points, %.0f s" % (len(points), len(keep), time.time() - t_start),
                      file=sys.stderr, flush=True)
        run.ks.ks_force_variant(None)
        families = {}
        if not args.no_families and args.kernel is None:
            run.fill("f32")
            fam = []
            for layout in ("bsf", "bsl"):
                fam.append(run.point((2, 4, 4, 2), 32, "f32", layout))
            for l in range(1, 11):
                fam.append(run.point((2 ** (l - 1), 2, 2, 2 ** (10 - l)), 4096, "f32", "bsl"))
            for dtype in ("f32", "bf16"):
                run.fill(dtype)
                for layout in ("bsf", "bsl"):
                    for p in ((1, 32, 32, 32), (32, 32, 32, 1)):
                        fam.append(run.point(p, 16384, dtype, layout))
                    for p in ((6, 64, 16, 8), (6, 16, 64, 8)):
                        fam.append(run.point(p, 25088, dtype, layout))
            for r in fam:
                fout.write(json.dumps(r) + "\n")
            # FP8 (E4M3 inputs, bf16 outputs): the MLP layers and every 7th
            # sweep pattern at both batches and layouts
            run.fill("fp8")
            fp8 = [run.point(p, 25088, "fp8", layout) for p in ((6, 64, 16, 8), (6, 16, 64, 8))
                   for layout in ("bsf", "bsl")]
            fp8_sweep = [run.point(p, batch, "fp8", layout) for batch in (4096, 25088) for layout in ("bsf", "bsl")
                         for p in sweep_patterns()[::7]]
            for r in fp8 + fp8_sweep:
                fout.write(json.dumps(r) + "\n")
            # bias + GELU epilogue on the MLP up-projection (768 -> 3072)
            epi = []
            for dtype in ("f32", "bf16"):
                run.fill(dtype)
                for layout in ("bsf", "bsl"):
                    epi.append(run.point((6, 64, 16, 8), 25088, dtype, layout, epilogue=True))
            for r in epi:
                fout.write(json.dumps(r) + "\n")
            run.fill("f32")
            bfly = [(2 ** (l - 1), 2, 2, 2 ** (10 - l)) for l in range(1, 11)]
            ch = [run.chain(bfly, 4096, "f32", "bsl")]
            for dtype in ("f32", "bf16"):
                run.fill(dtype)
                for layout in ("bsf", "bsl"):
                    ch.append(run.chain([(1, 32, 32, 32), (32, 32, 32, 1)], 16384, dtype, layout))
            run.fill("f32")
            bfly_more = [run.chain(bfly, 4096, "f32", "bsf"), run.chain(bfly, 4096, "f32", "bsl", fused=False)]
            for r in ch + bfly_more:
                fout.write(json.dumps(r) + "\n")

            def fam_summary(sel):
                return {"median_frac": float(np.median([r["frac"] for r in sel])),
                        "median_gbps": float(np.median([r["gbps"] for r in sel]))}
            families = {
                "tiny_(2,4,4,2)_B32_f32": fam_summary(fam[0:2]),
                "butterfly_N1024_B4096_f32_bsl": fam_summary(fam[2:12]),
                "monarch_B16384": fam_summary([r for r in fam[12:] if r["batch"] == 16384]),
                "mlp_768_3072_B25088": fam_summary([r for r in fam[12:] if r["batch"] == 25088]),
                "butterfly_10chain_B4096_f32_bsl_us": ch[0]["us"],
                "butterfly_10chain_B4096_f32": {
                    "bsl": {k: ch[0][k] for k in ("path", "us", "fused_lower_bound_us", "frac_fused_bound",
                                                  "frac_unfused")},
                    "bsf": {k: bfly_more[0][k] for k in ("path", "us", "fused_lower_bound_us", "frac_fused_bound",
                                                         "frac_unfused")},
                    "bsl_factor_by_factor_us": bfly_more[1]["us"]},
                "monarch_2chain_B16384_us": {"%s_%s" % (r["dtype"], r["layout"]): r["us"] for r in ch[1:]},
                "fp8_mlp_B25088": {"%s_%s" % (tuple(r["pattern"]), r["layout"]): {
                    "us": r["us"], "gbps": r["gbps"], "frac": r["frac"]} for r in fp8},
                "fp8_sweep_every7th": {"points": len(fp8_sweep),
                                       "median_frac": float(np.median([r["frac"] for r in fp8_sweep])),
                                       "median_gbps": float(np.median([r["gbps"] for r in fp8_sweep]))},
                "mlp_up_bias_gelu_B25088": {"%s_%s" % (r["dtype"], r["layout"]): {
                    "us": r["us"], "frac": r["frac"], "us_without_epilogue": next(
                        q["us"] for q in fam[12:] if q["batch"] == 25088 and tuple(q["pattern"]) == (6, 64, 16, 8)
                        and q["dtype"] == r["dtype"] and q["layout"] == r["layout"])} for r in epi},
            }
    fr = np.array([r["frac"] for r in points])
    # Dominant kernel instance: the largest share of one step, i.e. of one
    # call per sweep point (ms_per_step).  Its roofline figures are averages
    # over all of its timed calls, the way a profiler averages its dispatches:
    # each point contributes steps * calls_per_pass calls of the same
    # duration.
    per_k = {}
    for r in points:
        n = args.steps * r["calls_per_pass"]
        k = per_k.setdefault(r["kernel"], {"t": 0.0, "bytes": 0.0, "flops": 0.0, "calls": 0, "points": 0,
                                           "t_hbm": 0.0, "t_flop": 0.0, "dtype": r["dtype"], "t_step": 0.0})
        k["t"] += r["us"] * 1e-6 * n
        k["t_step"] += r["us"] * 1e-6
        k["bytes"] += r["bytes"] * n
        k["flops"] += r["flops"] * n
        k["calls"] += n
        k["points"] += 1
        k["t_hbm"] += r["bytes"] / HBM_BW * n
        k["t_flop"] += r["flops"] / PEAK[r["dtype"]] * n
    t_step = sum(v["t_step"] for v in per_k.values())
    t_timed = sum(v["t"] for v in per_k.values())
    dom_name, dom = max(per_k.items(), key=lambda kv: kv[1]["t_step"])
    if dom["t_hbm"] >= dom["t_flop"]:
        achieved = dom["bytes"] / dom["t"] / 1e9
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_BW / 1e9, "unit": "GB/s",
                    "frac": achieved / (HBM_BW / 1e9), "traffic": None}
    else:
        achieved = dom["flops"] / dom["t"] / 1e12
        roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK[dom["dtype"]] / 1e12, "unit": "TFLOP/s",
                    "frac": achieved / (PEAK[dom["dtype"]] / 1e12), "traffic": None}
    roofline["kernel"] = dom_name
    roofline["dominant_by"] = "largest share of one step (one call per sweep point)"
    roofline["points"] = dom["points"]
    roofline["timed_calls"] = dom["calls"]
    roofline["avg_launch_us"] = dom["t"] / dom["calls"] * 1e6
    roofline["algorithmic_bytes_per_launch"] = dom["bytes"] / dom["calls"]
    roofline["algorithmic_flops_per_launch"] = dom["flops"] / dom["calls"]
    roofline["share_of_step_time"] = dom["t_step"] / t_step
    roofline["share_of_timed_calls_time"] = dom["t"] / t_timed
    sha = kernel_sources_sha1()
    rec = traffic_record(dom_name, args.sample) if args.kernel is None and not args.eager else None
    if rec is not None:
        roofline["traffic"] = rec["traffic_bytes_per_launch"]
        roofline["traffic_unit"] = "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    ms_per_step = float(sum(r["us"] for r in points) * 1e-3)
    out = {
        "metric": METRIC,
        "value": float(np.median(fr)),
        "unit": "fraction of roofline (median over sweep points)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+bf16 (fp32 accumulate)",
        "data": "synthetic: X, K i.i.d. N(0,1), seeded",
        "config": {"workload": "KS pattern sweep a{1,2,4,8} x b,c{16,32,48,64,96,128} x d{1,2,4,8,16}, "
                               "abd,acd<=8192 (700 patterns) x B{4096,25088} x {fp32,bf16} x {BSF,BSL}",
                   "points": len(points), "sample_every": args.sample, "parallelism": "single GPU"},
        "forced_variant": args.variant if args.variant >= 0 else None,
        "only_kernel": args.kernel,
        "eager": args.eager,
        "sources_sha1": sha,
        "skipped_points": skipped,
        "median_gbps": float(np.median([r["gbps"] for r in points])),
        "median_tflops": float(np.median([r["tflops"] for r in points])),
        "frac_quantiles_10_25_50_75_90": [float(np.quantile(fr, q)) for q in (0.1, 0.25, 0.5, 0.75, 0.9)],
        "median_frac_by": {
            "%s_%s_B%d" % (dt, lay, B): float(np.median([r["frac"] for r in points
                                                        if r["dtype"] == dt and r["layout"] == lay and r["batch"] == B]))
            for dt in ("f32", "bf16") for lay in ("bsf", "bsl") for B in (4096, 25088)
            if any(r["dtype"] == dt and r["layout"] == lay and r["batch"] == B for r in points)},
        "roofline": roofline,
        "top_kernels": [{"kernel": k, "share_of_step_time": v["t_step"] / t_step,
                         "share_of_timed_calls_time": v["t"] / t_timed,
                         "points": v["points"], "avg_launch_us": v["t"] / v["calls"] * 1e6,
                         "gbps": v["bytes"] / v["t"] / 1e9}
                        for k, v in sorted(per_k.items(), key=lambda kv: -kv[1]["t_step"])[:5]],
        "top_kernels_by_timed_calls": [{"kernel": k, "share_of_timed_calls_time": v["t"] / t_timed,
                                        "points": v["points"], "avg_launch_us": v["t"] / v["calls"] * 1e6,
                                        "gbps": v["bytes"] / v["t"] / 1e9}
                                       for k, v in sorted(per_k.items(), key=lambda kv: -kv[1]["t"])[:3]],
        "families": families,
    }
    if any("launch_us_median" in r for r in points):
        fl = np.array([r["frac_launch_median"] for r in points if "frac_launch_median" in r])
        out["per_launch"] = {
            "what": "each point also timed call by call, each call between its own HIP event pair "
                    "(%d calls spread over the rotation); value uses the back-to-back graph-replay "
                    "time per call instead" % PER_LAUNCH_SAMPLES,
            "median_frac": float(np.median(fl)),
            "frac_quantiles_10_25_50_75_90": [float(np.quantile(fl, q)) for q in (0.1, 0.25, 0.5, 0.75, 0.9)]}
    # Every point, compact: pattern, batch, dtype, layout, time per call (us,
    # graph replay), GB/s, TFLOP/s, fraction of roofline, binding roof, and the
    # per-launch event median and IQR (us) when measured.
    out["points_fields"] = ["a", "b", "c", "d", "batch", "dtype", "layout", "us", "gbps", "tflops", "frac",
                            "bound", "launch_us_median", "launch_us_q1", "launch_us_q3"]
    out["points"] = [list(r["pattern"]) + [r["batch"], r["dtype"], r["layout"], round(r["us"], 3),
                                           round(r["gbps"], 1), round(r["tflops"], 3), round(r["frac"], 4),
                                           r["bound"], round(r.get("launch_us_median", float("nan")), 3),
                                           round(r.get("launch_us_iqr", [float("nan")] * 2)[0], 3),
                                           round(r.get("launch_us_iqr", [float("nan")] * 2)[1], 3)]
                     for r in points]
    if not args.no_cpu_baseline and args.kernel is None:
        out["cpu_baseline"] = cpu_baseline()
    out["wall_s"] = time.time() - t_start
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
