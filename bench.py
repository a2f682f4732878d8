#!/usr/bin/env python3
"""Benchmark of the Winograd hot path on one MI355X.

One step = one pass of the per-inference path over one batch: the
convolution (input transform -> T GEMMs -> output transform) of every layer in
the workload, plus the 2x2 pools of a stack.  The weight transform is done once
per weight set (offline in the method); it runs before the timed region and
is timed and reported on its own, and also as part of a second, full-step
figure.  Prints one JSON line.

Metric: effective GFLOP/s = direct-convolution FLOPs (2*N*K*C*9*Ho*Wo per layer)
divided by the step time, with eager launches (``--graph`` replays a HIP graph
of 10 steps instead; the eager and the other figure are both reported).  Also
reported:

* ``roofline``: the dominant launch's algorithmic bytes (or FLOPs) over its
  duration: primarily the cold median (after evicting L2 and the last-level
  cache), also the warm one from HIP events around a graph of back-to-back
  launches on its own stream; ``traffic`` is the HBM
  bytes per launch that rocprofv3's FETCH_SIZE / WRITE_SIZE counters measured
  for it (scaled by what they read for a plain device copy of known size), read
  from the committed counter summary under profiles/ -- or null when that
  summary was taken on other kernel sources than the ones built here.
* ``cpu_baseline``: the fp64 CPU oracle on this host's cores, on a bounded
  sample of the same workload.

``--pmc-summary FETCH_DIR WRITE_DIR`` turns two rocprofv3 --pmc runs of this
script (one with FETCH_SIZE, one with WRITE_SIZE, csv output) into that
committed summary.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

HBM_PEAK = 8.0e12          # B/s, MI355X HBM3E
FP32_MFMA_PEAK = 157.3e12  # FLOP/s, MI355X dense fp32 matrix
FP16_MFMA_PEAK = 2.5e15    # FLOP/s, MI355X dense fp16 / bf16 matrix
COPY_BYTES = 64 << 20      # size of the plain copy that calibrates the byte counters
EVICT_BYTES = 512 << 20    # read before each cold launch: twice the 256 MB last-level cache
HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_1903_01521_amd", "csrc")
PROFILES = os.path.join(HERE, "profiles")

# Kernel-name prefixes as rocprofv3 reports them, per kind of launch.
AXIS = {"w": 1, "h": 2}   # WINO_AXIS_W, WINO_AXIS_H

KERNEL_NAMES = {"filter": "void wino::k_filter", "fused": "void wino::k_fused", "lowc": "void wino::k_lowc",
                # the staged input transform: by tile rows, or by tiles for very wide images
                "input": "void wino::k_vrows|void wino::k_input", "gemm": "void wino::k_gemm",
                "output": "void wino::k_output", "maxpool": "void wino::k_maxpool2x2",
                "stages": "void wino::k_gemm", "stages16": "void wino::k_gemm16",
                # the split path on 16-bit operands: the 16-bit input transform, then
                # the GEMMs (16-bit MFMAs) with the output transform
                "split16": ("void wino::k_vrows|void wino::k_input16", "void wino::k_gemm_out"),
                "gemm16": "void wino::k_gemm16",
                # the split path's call: the input transform (by tile rows, or by 16-tile
                # patches for very wide images), then the GEMMs with the output transform
                "split": ("void wino::k_vrows|void wino::k_vblk", "void wino::k_gemm_out"),
                # the same on channel-last tensors: the NHWC input transform into the
                # blocked V, then the GEMMs storing y channel-last
                "split_nhwc": ("void wino::k_vrows_nhwc|void wino::k_input_nhwc4|void wino::k_input_nhwc",
                               "void wino::k_gemm_out"),
                # the fused kernel over channel slices, then the sum of the slices
                "fused_sliced": ("void wino::k_fused", "void wino::k_slice_sum")}


def kernel_label(kind: str) -> str:
    names = KERNEL_NAMES[kind]
    names = (names,) if isinstance(names, str) else names
    strip = lambda n: n[5:] if n.startswith("void ") else n
    return " + ".join(" or ".join(strip(a) for a in n.split("|")) for n in names)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def sources_hash() -> str:
    """sha256 over the HIP sources and host planner that define the kernels and launches."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*"))):
        if f.endswith((".hip", ".h", ".cpp")):
            h.update(os.path.basename(f).encode())
            h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def layer_numbers(N, L):
    """Sizes and algorithmic work of one layer (m x m tiles, alpha = m+2)."""
    if L.axis == "w":              # 1 x r filter: tiles of 1 x m, padding along W only
        Ho, Wo = L.H, L.W + 2 * L.pad - (L.r - 1)
        th, tw, T, taps = Ho, -(-Wo // L.m), 8, L.r
    elif L.axis == "h":            # r x 1 filter
        Ho, Wo = L.H + 2 * L.pad - (L.r - 1), L.W
        th, tw, T, taps = -(-Ho // L.m), Wo, 8, L.r
    else:
        Ho, Wo = L.H + 2 * L.pad - (L.r - 1), L.W + 2 * L.pad - (L.r - 1)
        th, tw, T, taps = -(-Ho // L.m), -(-Wo // L.m), (L.m + L.r - 1) ** 2, L.r * L.r
    P = N * th * tw
    f = dict(Ho=Ho, Wo=Wo, P=P, T=T)
    f["direct_flops"] = 2 * N * L.K * L.C * taps * Ho * Wo
    f["gemm_flops"] = 2 * T * P * L.C * L.K
    x_b, y_b, u_b = 4 * N * L.C * L.H * L.W, 4 * N * L.K * Ho * Wo, 4 * T * L.C * L.K
    v_b, m_b = 4 * T * P * L.C, 4 * T * P * L.K
    # minimum HBM bytes per kernel launch (what the method must move, padding excluded)
    f["bytes"] = {
        "filter": 4 * L.K * L.C * taps + u_b,
        "fused": x_b + u_b + y_b,
        "fused_sliced": x_b + u_b + y_b,
        "split": x_b + u_b + y_b,
        "split_nhwc": x_b + u_b + y_b,
        "lowc": x_b + u_b + y_b,
        "input": x_b + v_b,
        "gemm": v_b + u_b + m_b,
        "output": m_b + y_b,
        "maxpool": y_b + y_b // 4,
        # the three stages in one call (1-D and channel-last layers): x -> V -> M -> y
        "stages": x_b + 2 * v_b + u_b + 2 * m_b + y_b,
        # the same with 16-bit V and U (fp16 / bf16 GEMM operands)
        "stages16": x_b + v_b + u_b // 2 + 2 * m_b + y_b,
        # the split path on 16-bit operands: x and 16-bit U read, y written
        "split16": x_b + u_b // 2 + y_b,
        # the 16-bit GEMM stage alone: 16-bit V and U read, fp32 M written
        "gemm16": v_b // 2 + u_b // 2 + m_b,
        # the split path's two kernels: the input transform ("input"), then the
        # GEMMs with the output transform (V and U read, y written)
        "gemm_out": v_b + u_b + y_b,
        # the 16-bit input transform (16-bit V written)
        "input16": x_b + v_b // 2,
    }
    f["flops"] = {"fused": f["gemm_flops"], "fused_sliced": f["gemm_flops"], "split": f["gemm_flops"],
                  "split_nhwc": f["gemm_flops"], "gemm": f["gemm_flops"], "gemm_out": f["gemm_flops"],
                  "stages": f["gemm_flops"],
                  "stages16": f["gemm_flops"], "gemm16": f["gemm_flops"], "split16": f["gemm_flops"]}
    return f


def roofline(kind, nums, seconds):
    b = nums["bytes"].get(kind, 0)
    fl = nums["flops"].get(kind, 0)
    peak = FP16_MFMA_PEAK if kind in ("stages16", "gemm16", "split16") else FP32_MFMA_PEAK   # the GEMM's own operand type
    t_hbm = b / HBM_PEAK
    t_mfma = fl / peak
    if t_mfma >= t_hbm and fl > 0:
        ach = fl / seconds / 1e12
        return {"bound": "mfma", "achieved": round(ach, 3), "peak": peak / 1e12,
                "unit": "TFLOP/s", "frac": round(ach / (peak / 1e12), 4), "traffic": None,
                "algorithmic_flops": fl, "algorithmic_bytes": b}
    ach = b / seconds / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": round(ach / (HBM_PEAK / 1e9), 4), "traffic": None,
            "algorithmic_flops": fl, "algorithmic_bytes": b}


def traffic_file(workload: str, kind: str) -> str:
    """Counter summary of a workload's convolution kernel (fused, low-C), or of
    one stage of its staged path (input, gemm, output)."""
    if kind in ("fused", "fused_sliced", "split", "split_nhwc", "lowc"):
        return os.path.join(PROFILES, f"traffic_{workload}.txt")
    return os.path.join(PROFILES, f"traffic_{workload}_{kind}.txt")


def read_traffic(workload: str, kind: str):
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary, or None if there is none or it was taken on other sources."""
    path = traffic_file(workload, kind)
    if not os.path.exists(path):
        return None, "no counter summary"
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("sources_sha256") != sources_hash():
        return None, "kernel sources changed since the counters were taken"
    if kv.get("kind") != kind:
        return None, f"counter summary covers {kv.get('kind')}, not {kind}"
    return int(float(kv["traffic_bytes_per_launch"])), path


def pmc_rows(d: str):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = []
    for f in files:
        rows.extend(csv.DictReader(open(f)))
    return rows


def kernel_is(name: str, prefix: str) -> bool:
    """Whether a profiler kernel name is of the given kind: template instances
    carry their return type ("void wino::k_fused<...>(...)"), plain functions
    do not ("wino::k_gemm(...)").  A prefix "a|b" matches either kernel."""
    strip = lambda n: n[5:] if n.startswith("void ") else n
    n = strip(name)
    for base in (strip(p) for p in prefix.split("|")):
        if n.startswith(base) and n[len(base):len(base) + 1] in ("<", "("):
            return True
    return False


MFMA_COUNTERS = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "SQ_INSTS_MFMA", "GRBM_GUI_ACTIVE")


def mfma_summary(args):
    """Matrix-core work of a kind of launch from one rocprofv3 PMC run of this
    script with MFMA_COUNTERS.  On MI355X SQ_VALU_MFMA_BUSY_CYCLES reads 32 per
    v_mfma_f32_16x16x4_f32 (its issue cycles), so it measures work, not time;
    GRBM_GUI_ACTIVE is summed over the 8 XCDs.  Busy cycles over the active
    cycles of 1024 SIMDs give the utilisation while the launch ran (under the
    profiler, whose per-dispatch overhead weighs on short launches); the MFMA
    probe in the same run calibrates it (its value is its measured share of the
    published peak).  The instruction count checks the launch does exactly the
    MFMA work the algorithm needs, plus the padding of partial tile blocks."""
    from paper_1903_01521_amd import workloads as wl
    name = args.workload or wl.DEFAULT_BENCH
    w = wl.WORKLOADS[name]
    nums = [layer_numbers(w.N, L) for L in w.layers]
    kind = args.kind
    prefixes = KERNEL_NAMES[kind]
    prefixes = (prefixes,) if isinstance(prefixes, str) else prefixes
    rows = pmc_rows(args.mfma_summary)

    def mean(counter, pref):
        v = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == counter and kernel_is(r["Kernel_Name"], pref)]
        if not v:
            raise SystemExit(f"no {counter} rows for {pref} under {args.mfma_summary}")
        return float(np.mean(v)), len(v)

    simds = 256 * 4
    util = lambda busy, active: busy / (active / 8 * simds)
    pb, pn = mean("SQ_VALU_MFMA_BUSY_CYCLES", "void wino::k_mfma_probe")
    pg, _ = mean("GRBM_GUI_ACTIVE", "void wino::k_mfma_probe")
    kb = sum(mean("SQ_VALU_MFMA_BUSY_CYCLES", p)[0] for p in prefixes)
    kg = sum(mean("GRBM_GUI_ACTIVE", p)[0] for p in prefixes)
    ki = sum(mean("SQ_INSTS_MFMA", p)[0] for p in prefixes)
    kn = min(mean("SQ_INSTS_MFMA", p)[1] for p in prefixes)
    need = sum(f["flops"].get(kind, 0) for f in nums) / len(nums) / (2 * 16 * 16 * 4)
    fl = f" --flags {args.flags:#x}" if args.flags is not None else ""
    lines = [
        f"# MFMA work and utilisation of the {kind} launch on workload {name}, from one",
        "# rocprofv3 PMC run of bench.py on one MI355X (command below).",
        "#   mfma_insts: v_mfma_f32_16x16x4_f32 per launch, all waves (SQ_INSTS_MFMA);",
        "#   mfma_insts_algorithmic: the launch's algorithmic FLOPs / 2048;",
        "#   busy_cycles_per_inst: SQ_VALU_MFMA_BUSY_CYCLES / SQ_INSTS_MFMA;",
        "#   util_active: busy cycles / (GRBM_GUI_ACTIVE / 8 XCDs * 1024 SIMDs), and the",
        "#   same for the MFMA probe in this run (its share of the published peak).",
        "#   cd /tmp && export TMPDIR=/tmp",
        f"#   timeout -s KILL 90 rocprofv3 --pmc {' '.join(MFMA_COUNTERS)} --output-format csv -d <out>/mfma "
        f"-o run -- python3 <repo>/bench.py --workload {name}{fl} --steps 5 --warmup 1 --cpu-seconds 0 --no-graphs",
        f"#   python3 bench.py --workload {name}{fl} --kind {kind} --mfma-summary <out>/mfma",
        f"workload: {name}",
        f"kind: {kind}",
        f"kernels: {kernel_label(kind)}",
        f"sources_sha256: {sources_hash()}",
        f"dispatches: {kn}",
        f"mfma_insts: {ki:.0f}",
        f"mfma_insts_algorithmic: {need:.0f}",
        f"mfma_insts_over_algorithmic: {ki / need:.4f}",
        f"busy_cycles_per_inst: {kb / ki:.2f}",
        f"util_active: {util(kb, kg):.3f}",
        f"probe_util_active: {util(pb, pg):.3f} ({pn} dispatches)",
    ]
    text = "\n".join(lines) + "\n"
    if args.write_summary:
        with open(os.path.join(PROFILES, f"mfma_{name}_{kind}.txt"), "w") as fh:
            fh.write(text)
    print(text, end="")


def pmc_summary(args):
    """Summarise a FETCH_SIZE run and a WRITE_SIZE run of this script."""
    from paper_1903_01521_amd import workloads as wl
    name = args.workload or wl.DEFAULT_BENCH
    w = wl.WORKLOADS[name]
    nums = [layer_numbers(w.N, L) for L in w.layers]
    kind = args.kind
    prefixes = KERNEL_NAMES[kind]
    prefixes = (prefixes,) if isinstance(prefixes, str) else prefixes
    out = {}
    for counter, d in (("FETCH_SIZE", args.pmc_summary[0]), ("WRITE_SIZE", args.pmc_summary[1])):
        rows = [r for r in pmc_rows(d) if r["Counter_Name"] == counter]
        # the calibration launches: torch's elementwise negation over COPY_BYTES
        copy = [float(r["Counter_Value"]) for r in rows
                if "neg" in r["Kernel_Name"].lower() and int(r["Grid_Size"]) * 16 >= COPY_BYTES // 4]
        # a call of several kernels (the split path): the sum of their per-dispatch means
        per = [[float(r["Counter_Value"]) for r in rows if kernel_is(r["Kernel_Name"], p)] for p in prefixes]
        if not all(per) or not copy:
            raise SystemExit(f"{counter}: {[len(k) for k in per]} {kind} dispatches, {len(copy)} copy dispatches in {d}")
        out[counter] = (sum(float(np.mean(k)) for k in per), min(len(k) for k in per), float(np.median(copy)),
                        len(copy), sorted(set(r["Kernel_Name"] for r in rows
                                              if any(kernel_is(r["Kernel_Name"], p) for p in prefixes))))
    fk, fn_, fc, fcn, names = out["FETCH_SIZE"]
    wk, wn, wc, wcn, _ = out["WRITE_SIZE"]
    fscale = fc * 1024 / COPY_BYTES
    wscale = wc * 1024 / COPY_BYTES
    traffic = fk * 1024 / fscale + wk * 1024 / wscale
    alg = sum(f["bytes"][kind] for f in nums) / len(nums)
    fl = f" --flags {args.flags:#x}" if args.flags is not None else ""
    lines = [
        f"# HBM traffic per launch of the {kind} kernel on workload {name}",
        "# from two rocprofv3 PMC runs of bench.py on one MI355X (commands below), each",
        f"# counter scaled by what it reads for a plain streaming kernel over {COPY_BYTES} bytes.",
        "#   cd /tmp && export TMPDIR=/tmp",
        f"#   timeout -s KILL 60 rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/fetch -o run -- "
        f"python3 <repo>/bench.py --workload {name}{fl} --steps 20 --warmup 2 --cpu-seconds 0 --no-graphs",
        f"#   timeout -s KILL 60 rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/write -o run -- "
        f"python3 <repo>/bench.py --workload {name}{fl} --steps 20 --warmup 2 --cpu-seconds 0 --no-graphs",
        f"#   python3 bench.py --workload {name}{fl} --kind {kind} --pmc-summary <out>/fetch <out>/write",
        f"workload: {name}",
        f"kind: {kind}",
        f"kernels: {' | '.join(names)}",
        f"sources_sha256: {sources_hash()}",
        f"dispatches_fetch: {fn_}",
        f"dispatches_write: {wn}",
        f"fetch_kib_per_dispatch: {fk:.1f}",
        f"write_kib_per_dispatch: {wk:.1f}",
        f"copy_bytes: {COPY_BYTES}",
        f"copy_fetch_kib: {fc:.1f} (median of {fcn})",
        f"copy_write_kib: {wc:.1f} (median of {wcn})",
        f"fetch_scale: {fscale:.4f}",
        f"write_scale: {wscale:.4f}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        f"algorithmic_bytes_per_launch: {alg:.0f}",
        f"traffic_over_algorithmic: {traffic / alg:.3f}",
    ]
    text = "\n".join(lines) + "\n"
    if args.write_summary:
        with open(traffic_file(name, kind), "w") as fh:
            fh.write(text)
    print(text, end="")


def trace_summary(args):
    """Turn a rocprofv3 --kernel-trace --stats csv run of this script into the
    committed kernel-trace summary (per-kernel calls and durations)."""
    import re
    from paper_1903_01521_amd import workloads as wl
    name = args.workload or wl.DEFAULT_BENCH
    files = glob.glob(os.path.join(args.trace_summary, "**", "*kernel_stats.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one kernel_stats.csv under {args.trace_summary}, found {len(files)}")
    rows = list(csv.DictReader(open(files[0])))

    def short(n):
        n = re.sub(r"^void ", "", n)
        n = re.sub(r"\(.*$", "", n) if n.startswith("wino::") else n
        return n[:60] + ("..." if len(n) > 60 else "")
    fl = f" --flags {args.flags:#x}" if args.flags is not None else ""
    extra = f" {args.trace_args}" if args.trace_args else ""
    tag = f"_{args.tag}" if args.tag else ""
    lines = [f"# rocprofv3 kernel-trace summary: workload {name}{fl}",
             "# one MI355X; commands (on the GPU host; <repo> is the repository root):",
             "#   cd /tmp && export TMPDIR=/tmp",
             f"#   rocprofv3 --kernel-trace --stats --output-format csv -d <out>/prof -o run -- "
             f"python3 <repo>/bench.py --workload {name}{fl}{extra}",
             f"#   python3 <repo>/bench.py --workload {name}{fl} --trace-summary <out>/prof"
             + (f" --trace-args '{args.trace_args}'" if args.trace_args else "")
             + (f" --tag {args.tag}" if args.tag else ""),
             "# durations in ns; the calls include the warm-up, the timed steps and the",
             "# per-launch (warm, in-sequence and cold) timing runs of bench.py.",
             f"sources_sha256: {sources_hash()}",
             "",
             f"{'kernel':<64}{'calls':>7}{'avg_ns':>13}{'stddev':>11}{'min_ns':>9}{'max_ns':>9}"]
    for r in rows:
        lines.append(f"{short(r['Name']):<64}{int(r['Calls']):>7}{float(r['AverageNs']):>13.1f}"
                     f"{float(r['StdDev']):>11.1f}{int(r['MinNs']):>9}{int(r['MaxNs']):>9}")
    text = "\n".join(lines) + "\n"
    if args.write_summary:
        with open(os.path.join(PROFILES, f"kernel_trace_{name}{tag}.txt"), "w") as fh:
            fh.write(text)
    print(text, end="")


# Stage of a kernel of the step, by name (the first prefix that matches).
STAGE_OF = (("k_gemm_out", "gemm_out"), ("k_gemm16", "gemm16"), ("k_gemm", "gemm"), ("k_fused", "fused"),
            ("k_slice_sum", "slice_sum"), ("k_lowc", "lowc"), ("k_maxpool2x2", "maxpool"),
            ("k_vrows", "input"), ("k_vblk", "input"), ("k_input", "input"), ("k_output", "output"))
STAGE_MARKER = "FillFunctor"      # the torch fill that --stage-trace launches before every launch


def stage_table(args):
    """Per-layer, per-kernel durations of the step and each kernel's fraction of
    its own roofline, from a rocprofv3 --kernel-trace csv run of
    `bench.py --stage-trace DIR` (no GPU needed): the marker kernels split the
    trace into the step's launches; medians over the timed steps."""
    import re
    from paper_1903_01521_amd import workloads as wl
    d = args.stage_table
    meta = json.load(open(os.path.join(d, "launches.json")))
    name = meta["workload"]
    w = wl.WORKLOADS[name]
    nums = [layer_numbers(w.N, L) for L in w.layers]
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one kernel_trace.csv under {d}, found {len(files)}")
    rows = sorted(csv.DictReader(open(files[0])), key=lambda r: int(r["Dispatch_Id"]))
    launches = meta["launches"]                      # [[label, layer index], ...] of one step
    nl, steps = len(launches), meta["steps"]
    marks = [i for i, r in enumerate(rows) if STAGE_MARKER in r["Kernel_Name"]]
    if len(marks) < nl * steps:
        raise SystemExit(f"{len(marks)} marker kernels in the trace, expected at least {nl * steps}")
    marks = marks[-nl * steps:]
    per = {}                                         # (launch, kernel position) -> (name, [ns])
    for j, m0 in enumerate(marks):
        m1 = marks[j + 1] if j + 1 < len(marks) else len(rows)
        ks = [r for r in rows[m0 + 1:m1] if "wino::" in r["Kernel_Name"]]
        for q, r in enumerate(ks):
            key = (j % nl, q)
            nm = re.sub(r"\(.*$", "", re.sub(r"^void ", "", r["Kernel_Name"]))
            nm = nm.replace("wino::", "").replace(" ", "")
            per.setdefault(key, (nm, []))[1].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    prec = (meta["flags"] & 0x30) != 0               # 16-bit GEMM operands
    fl = f" --flags {meta['flags']:#x}" if meta["flags"] else ""
    lines = [f"# Per-layer, per-kernel durations of the timed step: workload {name}{fl}",
             "# one MI355X; each kernel's median over the timed steps (eager launches in",
             "# sequence, so every kernel runs after its real predecessor), and its fraction",
             "# of its own roofline from the algorithmic FLOPs or bytes of its stage",
             "# (input/output transforms and pools: HBM bytes; GEMMs: MFMA FLOPs or HBM",
             "# bytes, whichever bounds them; peaks 157.3 TFLOP/s fp32, 8 TB/s).",
             "# commands (on the GPU host; <repo> is the repository root):",
             "#   cd /tmp && export TMPDIR=/tmp",
             f"#   rocprofv3 --kernel-trace --output-format csv -d <out>/st -o run -- python3 <repo>/bench.py "
             f"--workload {name}{fl} --steps {steps} --warmup {meta['warmup']} --stage-trace <out>/st",
             f"#   python3 <repo>/bench.py --stage-table <out>/st",
             f"sources_sha256: {sources_hash()}",
             "",
             f"{'launch':<10}{'layer':<22}{'kernel':<34}{'stage':<10}{'med_us':>9}{'p10':>9}{'p90':>9}"
             f"  {'bound':<5}{'achieved':>10} {'unit':<8}{'frac':>7}"]
    total_ns = 0.0
    conv_ns = [0.0] * len(w.layers)
    for (li, q) in sorted(per):
        nm, ns = per[(li, q)]
        label, layer = launches[li]
        L, f = w.layers[layer], nums[layer]
        base = nm.split("<")[0]
        stage = next((st for pre, st in STAGE_OF if base.startswith(pre)), None)
        if stage == "input" and prec:
            stage = "input16"
        med, p10, p90 = float(np.median(ns)), float(np.percentile(ns, 10)), float(np.percentile(ns, 90))
        total_ns += med
        if stage != "maxpool":
            conv_ns[layer] += med
        shape = f"{L.C}->{L.K} @{L.H}x{L.W} m{L.m}" + (f" r{L.r}" if L.r != 3 else "")
        rf = roofline(stage, f, med * 1e-9) if stage in f["bytes"] else None
        if stage == "maxpool":             # the pool reads this layer's y and writes a quarter of it
            rf = roofline("maxpool", f, med * 1e-9)
        tail = (f"  {rf['bound']:<5}{rf['achieved']:>10} {rf['unit']:<8}{rf['frac']:>7.3f}" if rf
                else "  -")
        lines.append(f"{label:<10}{shape:<22}{nm[:33]:<34}{stage or '-':<10}{med / 1e3:>9.1f}{p10 / 1e3:>9.1f}"
                     f"{p90 / 1e3:>9.1f}{tail}")
    lines.append("")
    lines.append(f"step: {total_ns / 1e3:.1f} us (sum of the kernel medians)")
    for i, (L, f) in enumerate(zip(w.layers, nums)):
        if conv_ns[i] > 0:
            lines.append(f"L{i} conv: {conv_ns[i] / 1e3:.1f} us, {f['direct_flops'] / conv_ns[i] / 1e3:.1f} "
                         f"TFLOP/s effective (direct-conv FLOPs)")
    text = "\n".join(lines) + "\n"
    if args.write_summary:
        tag = f"_{args.tag}" if args.tag else ""
        with open(os.path.join(PROFILES, f"stage_table_{name}{tag}.txt"), "w") as fh:
            fh.write(text)
    print(text, end="")


# Layers whose algorithm choice the planner table records: the single 3x3
# layers, one layer of the ResNet stage, and the VGG-16 layers at N=1 and N=32.
PLANNER_WORKLOADS = ("f2_n1_c32_k32_56x56", "f4_n1_c64_k64_112x112", "f4_n1_c48_k48_57x57",
                     "f4_resnet_stage_n8_c128_28x28", "vgg16_stack_n1", "vgg16_stack_n32",
                     "f4_n64_c256_k256_56x56", "f4_lowc_n64_c3_k64_224x224", "f4_lowc_n1_c3_k64_224x224")
PLANNER_TABLE = os.path.join(PROFILES, "planner_table.txt")


def planner_layers():
    """Unique (N, C, H, W, K, pad, m) of the layers PLANNER_WORKLOADS run."""
    from paper_1903_01521_amd import workloads as wl
    seen, out = set(), []
    for name in PLANNER_WORKLOADS:
        w = wl.WORKLOADS[name]
        for L in w.layers:
            key = (w.N, L.C, L.H, L.W, L.K, L.pad, L.m)
            if key not in seen:
                seen.add(key)
                out.append(key)
    return out


def read_planner_table(path=PLANNER_TABLE):
    """Rows of the committed planner table: dict per layer with the shape, the
    measured time (us) of every algorithm the library accepted for it, and
    AUTO's choice when the table was taken."""
    rows = []
    for line in open(path):
        if line.startswith("#") or not line.strip() or line.startswith("N ") or ":" in line.split()[0]:
            continue
        f = line.split()
        shape = tuple(int(v) for v in f[:7])
        times = {}
        for kv in f[7:-2]:
            k, v = kv.split("=")
            times[k] = float(v)
        rows.append(dict(shape=shape, times=times, best=f[-2], auto=f[-1]))
    return rows


def planner_candidate_name(algo: int, nsl: int) -> str:
    from paper_1903_01521_amd import binding as B
    base = {B.WINO_ALGO_FUSED: "fused", B.WINO_ALGO_SPLIT: "split", B.WINO_ALGO_STAGED: "staged",
            B.WINO_ALGO_LOWC: "lowc"}[algo]
    return f"{base}_s{nsl}" if nsl > 1 else base


def planner_table(args):
    """Time every algorithm the library accepts on each planner layer (graph
    of back-to-back calls, median of replays) and record AUTO's choice."""
    import torch
    from paper_1903_01521_amd import binding as B
    B.lib()
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(0)
    lines = ["# Planner table: per-layer time (us, one wino_conv2d call, HIP graph of 10 back-to-back",
             "# calls, median of 5 replays) of every algorithm the library accepts for the layer",
             "# (fused: the planner's fused variant without channel slices; fused_sN: with N slices;",
             "# split; staged; lowc), the fastest, and AUTO's choice (wino_plan_r) when taken.",
             "# one MI355X; command (on the GPU host, from the repository root):",
             "#   python3 bench.py --planner-table --write-summary",
             f"sources_sha256: {sources_hash()}",
             "N C H W K pad m  times...  best auto"]

    def time_us(fn):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(2):
                B.check(fn(torch.cuda.current_stream().cuda_stream), "warm-up")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(10):
                B.check(fn(torch.cuda.current_stream().cuda_stream), "capture")
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(5):
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3 / 10)
        del g
        return float(np.median(ts))

    for (N, C, H, W, K, pad, m) in planner_layers():
        x = torch.from_numpy(rng.standard_normal((N, C, H, W)).astype(np.float32)).to(dev)
        g = torch.from_numpy((rng.standard_normal((K, C, 3, 3)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)).to(dev)
        U = torch.empty(B.wino_filter_bytes(C, K, m) // 4, dtype=torch.float32, device=dev)
        B.check(B.wino_filter_transform(g, U, C, K, m), "wino_filter_transform")
        Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
        y = torch.empty((N, K, Ho, Wo), dtype=torch.float32, device=dev)
        st, algo, nsl = B.wino_plan_r(N, C, H, W, K, pad, m, 3, 0)
        B.check(st, "wino_plan_r")
        auto = planner_candidate_name(algo, nsl)
        cands = [("fused", B.WINO_ALGO_FUSED)] + [(f"fused_s{n}", B.WINO_ALGO_FUSED | B.WINO_CSLICES(n))
                                                  for n in (2, 4)] + [
            ("split", B.WINO_ALGO_SPLIT), ("staged", B.WINO_ALGO_STAGED), ("lowc", B.WINO_ALGO_LOWC)]
        times = {}
        for cname, fl in cands:
            wsb = B.wino_workspace_bytes(N, C, H, W, K, pad, m, fl)
            if wsb == 2**64 - 1:
                continue
            if cname.startswith("fused_s"):
                stc, a2, n2 = B.wino_plan_r(N, C, H, W, K, pad, m, 3, fl)
                if stc != 0 or n2 <= 1:
                    continue
            ws = torch.empty(max(wsb // 4, 1), dtype=torch.float32, device=dev)
            fn = (lambda sp, fl=fl, ws=ws, wsb=wsb:
                  B.wino_conv2d(x, U, y, N, C, H, W, K, pad, m, fl, ws if wsb else None, wsb, sp))
            times[cname] = time_us(fn)
            del ws
        best = min(times, key=times.get)
        log(f"planner N={N} C={C} {H}x{W} K={K} m={m}: " +
            " ".join(f"{k}={v:.1f}" for k, v in times.items()) + f"  best {best} auto {auto}")
        lines.append(f"{N} {C} {H} {W} {K} {pad} {m}  " + " ".join(f"{k}={v:.1f}" for k, v in times.items())
                     + f"  {best} {auto}")
        del x, g, U, y
        torch.cuda.empty_cache()
    text = "\n".join(lines) + "\n"
    if args.write_summary:
        with open(PLANNER_TABLE, "w") as fh:
            fh.write(text)
    print(text, end="")


def sleep_calibration(stream) -> float:
    """GPU cycles per millisecond of torch's spin kernel (torch.cuda._sleep)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    n = 2_000_000
    e0.record(stream)
    torch.cuda._sleep(n)
    e1.record(stream)
    torch.cuda.synchronize()
    return n / max(e0.elapsed_time(e1), 1e-3)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--algo", choices=["auto", "fused", "staged"], default="auto")
    ap.add_argument("--flags", type=lambda s: int(s, 0), default=None,
                    help="explicit wino_conv2d flags (overrides --algo)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of a HIP graph holding 10 steps (K a multiple of 10) "
                         "instead of eager launches")
    ap.add_argument("--eager", action="store_true", help="eager launches (the default)")
    ap.add_argument("--no-graphs", action="store_true",
                    help="capture no HIP graph at all (per-kernel timing from eager launches); "
                         "for counter-collection runs")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU time budget of the oracle baseline (0 disables it)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc csv runs (no GPU needed)")
    ap.add_argument("--mfma-summary", metavar="DIR",
                    help="summarise a rocprofv3 --pmc run with the MFMA counters (matrix-core utilisation)")
    ap.add_argument("--trace-summary", metavar="DIR",
                    help="summarise a rocprofv3 --kernel-trace --stats csv run (no GPU needed)")
    ap.add_argument("--trace-args", default="", help="with --trace-summary: the profiled run's other arguments")
    ap.add_argument("--tag", default="", help="with --trace-summary: suffix of the summary's file name")
    ap.add_argument("--kind", default="fused", help="kernel kind the --pmc-summary covers")
    ap.add_argument("--write-summary", action="store_true",
                    help="with --pmc-summary: also write it to profiles/traffic_<workload>.txt")
    ap.add_argument("--stage-trace", metavar="DIR",
                    help="run only the step (W + K times), a marker kernel before every launch, and write "
                         "DIR/launches.json; for a rocprofv3 --kernel-trace run that --stage-table reads")
    ap.add_argument("--stage-table", metavar="DIR",
                    help="per-layer, per-kernel durations and stage rooflines from such a run (no GPU needed)")
    ap.add_argument("--planner-table", action="store_true",
                    help="time every algorithm on the planner's reference layers (profiles/planner_table.txt)")
    args = ap.parse_args()

    if args.pmc_summary:
        pmc_summary(args)
        return
    if args.mfma_summary:
        mfma_summary(args)
        return
    if args.trace_summary:
        trace_summary(args)
        return
    if args.stage_table:
        stage_table(args)
        return

    if args.planner_table:
        planner_table(args)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1903_01521_amd import binding as B
    from paper_1903_01521_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()   # fails loudly if libwino.so is not built

    name = args.workload or wl.DEFAULT_BENCH
    w = wl.WORKLOADS[name]
    N = w.N
    flags = args.flags if args.flags is not None else {
        "auto": B.WINO_ALGO_AUTO, "fused": B.WINO_ALGO_FUSED, "staged": B.WINO_ALGO_STAGED}[args.algo]
    staged = (flags & B.WINO_ALGO_MASK) == B.WINO_ALGO_STAGED
    prec = flags & B.WINO_PREC_MASK       # 16-bit GEMM operands (reduced precision, opt-in)
    if prec:
        staged = False                    # the three stages run inside one wino_conv2d call

    x, gs = wl.generate(w)
    dev = torch.device("cuda:0")
    # channel-last workloads get x as [N][H][W][C] (outside the timed region)
    hx = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 2, 3, 1)) if w.first.nhwc else x).to(dev)
    hg = [torch.from_numpy(g).to(dev) for g in gs]
    nums = [layer_numbers(N, L) for L in w.layers]

    # Device buffers, all allocated before timing.
    Us, ys, pools, wss, Vs, Ms = [], [], [], [], [], []
    H, W = w.first.H, w.first.W
    for L, f in zip(w.layers, nums):
        assert (L.H, L.W) == (H, W)
        if L.axis:
            ub = B.wino_filter_bytes_1d(L.C, L.K, L.m, L.r)
        elif prec:
            ub = B.wino_filter_bytes_p(L.C, L.K, L.m, prec)
        else:
            ub = B.wino_filter_bytes_r(L.C, L.K, L.m, L.r)
        Us.append(torch.empty(ub // 4, dtype=torch.float32, device=dev))
        ys.append(torch.empty((N, f["Ho"], f["Wo"], L.K) if L.nhwc else (N, L.K, f["Ho"], f["Wo"]),
                              dtype=torch.float32, device=dev))
        if L.nhwc:
            wsb = B.wino_workspace_bytes_nhwc(N, L.C, L.H, L.W, L.K, L.pad, L.m, flags)
        elif L.axis:
            wsb = B.wino_workspace_bytes_1d(N, L.C, L.H, L.W, L.K, L.pad, L.m, L.r, AXIS[L.axis], flags)
        else:
            wsb = B.wino_workspace_bytes_r(N, L.C, L.H, L.W, L.K, L.pad, L.m, L.r, flags)
        if wsb == 2**64 - 1:
            raise SystemExit(f"{name} layer {len(wss)} ({L.C}->{L.K} at {L.H}x{L.W}, m={L.m}, r={L.r}): "
                             f"the library rejects flags {flags:#x} for it (workspace size query failed)")
        wss.append((torch.empty(max(wsb // 4, 1), dtype=torch.float32, device=dev), wsb))
        if staged and not L.axis and not L.nhwc:
            Vs.append(torch.empty(B.wino_input_tf_bytes_r(N, L.C, L.H, L.W, L.pad, L.m, L.r) // 4,
                                  dtype=torch.float32, device=dev))
            Ms.append(torch.empty(B.wino_gemm_out_bytes_r(N, L.K, L.H, L.W, L.pad, L.m, L.r) // 4,
                                  dtype=torch.float32, device=dev))
        else:
            Vs.append(None)
            Ms.append(None)
        H, W = f["Ho"], f["Wo"]
        if L.pool:
            pools.append(torch.empty((N, L.K, H // 2, W // 2), dtype=torch.float32, device=dev))
            H, W = H // 2, W // 2
        else:
            pools.append(None)

    def launches():
        """The step as a list of (label, layer index, kind, fn(stream))."""
        out = []
        a = hx
        for i, L in enumerate(w.layers):
            relu = B.WINO_FLAG_RELU if L.relu else 0
            if L.nhwc:                     # channel-last layer: split, or the three stages, in one call
                ws, wsb = wss[i]
                out.append((f"L{i}.filter", i, "filter", (lambda sp, i=i, L=L: B.wino_filter_transform(
                    hg[i], Us[i], L.C, L.K, L.m, sp))))
                # the plan's workspace tells which: the split path's blocked V, or V and M
                split_wsb = B.wino_workspace_bytes_nhwc(N, L.C, L.H, L.W, L.K, L.pad, L.m,
                                                        (flags & ~B.WINO_ALGO_MASK) | B.WINO_ALGO_SPLIT)
                kind = "split_nhwc" if wsb == split_wsb and (flags & B.WINO_ALGO_MASK) != B.WINO_ALGO_STAGED else "stages"
                out.append((f"L{i}.conv", i, kind, (lambda sp, i=i, L=L, a=a, relu=relu, ws=ws, wsb=wsb:
                                                         B.wino_conv2d_nhwc(a, Us[i], ys[i], N, L.C, L.H, L.W, L.K,
                                                                            L.pad, L.m, flags | relu, ws, wsb, sp))))
                a = ys[i]
                continue
            if L.axis:                     # 1-D layer: the three stages in one call
                ws, wsb = wss[i]
                out.append((f"L{i}.filter", i, "filter", (lambda sp, i=i, L=L: B.wino_filter_transform_1d(
                    hg[i], Us[i], L.C, L.K, L.m, L.r, sp))))
                out.append((f"L{i}.conv", i, "stages", (lambda sp, i=i, L=L, a=a, relu=relu, ws=ws, wsb=wsb:
                                                         B.wino_conv2d_1d(a, Us[i], ys[i], N, L.C, L.H, L.W, L.K,
                                                                          L.pad, L.m, L.r, AXIS[L.axis],
                                                                          flags | relu, ws, wsb, sp))))
                a = ys[i]
                continue
            if prec:
                out.append((f"L{i}.filter", i, "filter", (lambda sp, i=i, L=L: B.wino_filter_transform_p(
                    hg[i], Us[i], L.C, L.K, L.m, prec, sp))))
            else:
                out.append((f"L{i}.filter", i, "filter",
                            (lambda sp, i=i, L=L: B.wino_filter_transform_r(hg[i], Us[i], L.C, L.K, L.m, L.r, sp))))
            if staged and not prec:
                out.append((f"L{i}.input", i, "input", (lambda sp, i=i, L=L, a=a: B.wino_input_transform_r(
                    a, Vs[i], N, L.C, L.H, L.W, L.pad, L.m, L.r, sp))))
                out.append((f"L{i}.gemm", i, "gemm", (lambda sp, i=i, L=L: B.wino_batched_gemm_r(
                    Us[i], Vs[i], Ms[i], N, L.C, L.H, L.W, L.K, L.pad, L.m, L.r, sp))))
                out.append((f"L{i}.output", i, "output", (lambda sp, i=i, L=L, relu=relu: B.wino_output_transform_r(
                    Ms[i], ys[i], N, L.K, L.H, L.W, L.pad, L.m, L.r, relu, sp))))
            else:
                ws, wsb = wss[i]
                st, algo, nsl = B.wino_plan_r(N, L.C, L.H, L.W, L.K, L.pad, L.m, L.r, flags | relu)
                B.check(st, "wino_plan_r")
                if prec:
                    kind = "split16" if algo == B.WINO_ALGO_SPLIT else "stages16"
                else:
                    kind = {B.WINO_ALGO_LOWC: "lowc", B.WINO_ALGO_SPLIT: "split"}.get(
                        algo, "fused_sliced" if nsl > 1 else "fused")
                out.append((f"L{i}.conv", i, kind, (lambda sp, i=i, L=L, a=a, relu=relu, ws=ws, wsb=wsb:
                                                       B.wino_conv2d_r(a, Us[i], ys[i], N, L.C, L.H, L.W, L.K,
                                                                       L.pad, L.m, L.r, flags | relu,
                                                                     ws if wsb else None, wsb, sp))))
            a = ys[i]
            if L.pool:
                out.append((f"L{i}.pool", i, "maxpool", (lambda sp, i=i, L=L, a=a: B.wino_maxpool2x2(
                    a, pools[i], N, L.K, nums[i]["Ho"], nums[i]["Wo"], sp))))
                a = pools[i]
        return out

    step = launches()

    def run(fns):
        sp = torch.cuda.current_stream().cuda_stream
        for label, fn in fns:
            st = fn(sp)
            if st != 0:
                raise RuntimeError(f"{label}: {B.wino_status_string(st)}")

    # The timed step: every launch but the weight transforms, which run once
    # before it (and in a second, full-step timing below).
    step_fns = [(label, fn) for label, _, kind, fn in step if kind != "filter"]
    filter_fns = [(label, fn) for label, _, kind, fn in step if kind == "filter"]
    full_fns = [(label, fn) for label, _, _, fn in step]

    def capture(fns, reps=1):
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            run(fns)                 # one eager pass on the capture stream first
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            for _ in range(reps):
                run(fns)
        torch.cuda.synchronize()
        return g

    if args.stage_trace:
        # The step alone, a torch fill (the marker) before every launch; the
        # launch list goes beside the trace for --stage-table.
        layer_of = {label: i for label, i, kind, _ in step if kind != "filter"}
        mk = torch.empty(1024, dtype=torch.float32, device=dev)
        run(filter_fns)
        for _ in range(args.warmup + args.steps):
            for label, fn in step_fns:
                mk.fill_(1.0)
                run([(label, fn)])
        torch.cuda.synchronize()
        os.makedirs(args.stage_trace, exist_ok=True)
        with open(os.path.join(args.stage_trace, "launches.json"), "w") as fh:
            json.dump({"workload": name, "flags": flags, "steps": args.steps, "warmup": args.warmup,
                       "launches": [[label, layer_of[label]] for label, _ in step_fns]}, fh)
        print(f"stage trace: {args.warmup + args.steps} steps of {len(step_fns)} launches", flush=True)
        return

    stream = torch.cuda.current_stream()
    GS = 10
    use_graph = args.graph and not args.eager and not args.no_graphs
    if use_graph and args.steps % GS:
        raise SystemExit(f"--graph needs --steps to be a multiple of {GS}")
    graph = capture(step_fns, reps=GS) if use_graph else None

    run(filter_fns)                      # U of every layer, once per weight set
    for _ in range(args.warmup):
        run(step_fns)
    torch.cuda.synchronize()

    # Timed region: exactly K steps, synchronised on both sides.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    if graph is None:
        for _ in range(args.steps):
            run(step_fns)
    else:
        for _ in range(args.steps // GS):
            graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall1 = time.perf_counter()
    ms_step = e0.elapsed_time(e1) / args.steps

    # The full step with the weight transforms, eager, for reference (outside
    # the timed region above).
    full_steps = max(1, min(args.steps, 200))
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(full_steps):
        run(full_fns)
    e1.record(stream)
    torch.cuda.synchronize()
    full_ms = e0.elapsed_time(e1) / full_steps

    # The other launch mode of the same step, for reference (outside the timed region).
    ref_steps = 20 * GS
    torch.cuda.synchronize()
    if args.no_graphs:
        eager_ms, graph_ms = ms_step, None
    elif graph is None:
        g_ref = capture(step_fns, reps=GS)
        e0.record(stream)
        for _ in range(ref_steps // GS):
            g_ref.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        eager_ms, graph_ms = ms_step, e0.elapsed_time(e1) / ref_steps
        g_ref = None
    else:
        e0.record(stream)
        for _ in range(ref_steps):
            run(step_fns)
        e1.record(stream)
        torch.cuda.synchronize()
        eager_ms, graph_ms = e0.elapsed_time(e1) / ref_steps, ms_step

    # Per-kernel average launch durations: for each launch of the step, a graph
    # of R back-to-back launches of it alone (no host launch gaps), timed under
    # HIP events on the stream the kernels run on.  Repeating a kernel alone lets
    # inputs that fit the 256 MB last-level cache stay there; the in-sequence
    # durations below show what each kernel takes after its real predecessors.
    R = 20
    reps = max(1, min(args.steps // 10, 50))
    per_launch, per_launch_spread = [], []
    for label, _, _, fn in step:
        if args.no_graphs:
            g = None
            def launch_r(fn=fn, label=label):
                run([(label, fn)] * R)
        else:
            g = capture([(label, fn)], reps=R)
            launch_r = g.replay
        launch_r()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0.record(stream)
            launch_r()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / R)
        per_launch.append(float(np.median(ts)))
        per_launch_spread.append((float(np.percentile(ts, 10)), float(np.percentile(ts, 90))))
        launch_r = g = None

    # In-sequence durations: HIP events around every launch of KP more eager
    # steps.  The GPU is first held in a spin kernel while the host enqueues all
    # KP steps, so the launches then run back to back with no host gaps, each
    # after its real predecessors (cache state as in the timed region).  Each
    # figure includes the launch's dispatch latency (~3 us), which back-to-back
    # launches of one kernel hide.
    cyc_per_ms = sleep_calibration(stream)
    KP = max(1, min(args.steps, 300 // len(step)))
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in step] for _ in range(KP)]
    sp = stream.cuda_stream
    hold_ms = 20.0
    for _ in range(3):
        torch.cuda.synchronize()
        torch.cuda._sleep(int(hold_ms * cyc_per_ms))
        h0 = time.perf_counter()
        for k in range(KP):
            for (label, _, _, fn), (a0, a1) in zip(step, evs[k]):
                a0.record(stream)
                st = fn(sp)
                a1.record(stream)
                if st != 0:
                    raise RuntimeError(f"{label}: {B.wino_status_string(st)}")
        enqueue_ms = (time.perf_counter() - h0) * 1e3
        torch.cuda.synchronize()
        gapless = enqueue_ms < 0.8 * hold_ms
        if gapless:
            break
        hold_ms = 2.5 * enqueue_ms
    in_seq = [float(np.mean([evs[k][i][0].elapsed_time(evs[k][i][1]) for k in range(KP)]))
              for i in range(len(step))]
    torch.cuda.synchronize()

    # Cold durations: before a launch a 512 MB read (a reduction into one
    # float) evicts L2 and the last-level cache, so the launch reads its inputs
    # from HBM; the same launch then runs once more, warm.  Both are timed with
    # HIP events in the enqueue-while-held scheme above; the cold figure is the
    # graph-timed duration plus the cold-minus-warm difference of those events,
    # so the events' own dispatch latency cancels.
    KC = max(3, min(10, 300 // len(step)))
    evict_src = torch.empty(EVICT_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    evict_dst = torch.empty((), dtype=torch.float32, device=dev)
    cev = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in step] for _ in range(KC)]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(20.0 * cyc_per_ms))
    for k in range(KC):
        for i, (label, _, _, fn) in enumerate(step):
            ev = cev[k][i]
            torch.sum(evict_src, dim=0, out=evict_dst)
            ev[0].record(stream)
            st = fn(sp)
            ev[1].record(stream)
            st |= fn(sp)
            ev[2].record(stream)
            if st != 0:
                raise RuntimeError(f"{label}: {B.wino_status_string(st)}")
    torch.cuda.synchronize()
    cold = []
    for i in range(len(step)):
        c = [cev[k][i][0].elapsed_time(cev[k][i][1]) for k in range(KC)]
        wm = float(np.median([cev[k][i][1].elapsed_time(cev[k][i][2]) for k in range(KC)]))
        cold.append([per_launch[i] + ck - wm for ck in c])
    del evict_src

    total_by = {}
    for (label, li, kind, _), t in zip(step, per_launch):
        total_by[kind] = total_by.get(kind, 0.0) + t
    # the dominant launch of the timed step (weight transforms excluded)
    dom = max((i for i, (_, _, k, _) in enumerate(step) if k != "filter"), key=lambda i: per_launch[i])
    dlabel, dlayer, dkind, _ = step[dom]
    cold_med = [float(np.median(c)) for c in cold]
    # primary: the cold median (inputs from HBM, not from a cache a repeated
    # launch warmed); the warm back-to-back figure beside it
    roof = roofline(dkind, nums[dlayer], cold_med[dom] / 1e3)
    roof["kernel"] = f"{dlabel} ({kernel_label(dkind)})"
    roof["avg_us"] = round(cold_med[dom] * 1e3, 3)
    roof["timing"] = "cold median (L2 and last-level cache evicted before each launch)"
    roof["avg_us_warm"] = round(per_launch[dom] * 1e3, 3)
    roof["frac_warm"] = roofline(dkind, nums[dlayer], per_launch[dom] / 1e3)["frac"]
    traffic, src = read_traffic(name, dkind) if len(w.layers) == 1 else (None, "multi-layer workload")
    roof["traffic"] = traffic
    roof["traffic_source"] = os.path.relpath(src, HERE) if traffic is not None else src

    # Plain streaming kernel of known size (reads COPY_BYTES, writes COPY_BYTES:
    # torch's elementwise negation): calibrates the HBM byte counters of the
    # rocprofv3 PMC runs of this script.  It runs outside every timed region.
    cs = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).uniform_()
    cd = torch.empty_like(cs)
    for _ in range(3):
        torch.neg(cs, out=cd)
    e0.record(stream)
    torch.neg(cs, out=cd)
    e1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * COPY_BYTES / (e0.elapsed_time(e1) / 1e3) / 1e9
    del cs, cd

    # Sustained fp32 matrix-core rate (the library's probe: 2048 waves of
    # independent MFMA chains), best of five launches, outside every timed region.
    probe_iters = 4096
    probe_out = torch.empty(2048, dtype=torch.float32, device=dev)
    B.check(B.wino_probe_mfma_f32(probe_iters, probe_out, stream), "wino_probe_mfma_f32")
    probe_ms = []
    for _ in range(5):
        e0.record(stream)
        B.check(B.wino_probe_mfma_f32(probe_iters, probe_out, stream), "wino_probe_mfma_f32")
        e1.record(stream)
        torch.cuda.synchronize()
        probe_ms.append(e0.elapsed_time(e1))
    if not bool((probe_out == 32.0 * probe_iters).all()):
        raise RuntimeError("MFMA probe check values are wrong")
    mfma_tflops = B.wino_probe_mfma_f32_flops(probe_iters) / (min(probe_ms) / 1e3) / 1e12

    direct = sum(f["direct_flops"] for f in nums)
    value = direct / (ms_step / 1e3) / 1e9
    filter_us = [t * 1e3 for (_, _, k, _), t in zip(step, per_launch) if k == "filter"]

    result = {
        "metric": "effective GFLOP/s (direct-conv FLOPs) per 3x3 layer + % of HBM/MFMA roofline",
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {0: "f32", B.WINO_PREC_F16: "f16 operands, f32 accumulate",
                  B.WINO_PREC_BF16: "bf16 operands, f32 accumulate"}[prec],
        "data": "synthetic",
        "config": {"workload": name, "N": N, "layers": len(w.layers),
                   "C": w.first.C, "K": w.first.K, "H": w.first.H, "W": w.first.W,
                   "m": w.first.m, "r": w.first.r, "axis": w.first.axis or "2d",
                   "layout": "nhwc" if w.first.nhwc else "nchw", "pad": w.first.pad,
                   "flags": hex(flags),
                   "launch": "eager" if graph is None else "hip_graph", "parallelism": "none"},
        "roofline": roof,
        "per_launch_us": {lbl: round(t * 1e3, 3) for (lbl, *_), t in zip(step, per_launch)},
        "per_kind_us": {k: round(t * 1e3, 3) for k, t in total_by.items()},
        "per_launch_in_sequence_us": {lbl: round(t * 1e3, 3) for (lbl, *_), t in zip(step, in_seq)},
        "in_sequence_timing": {"steps": KP, "host_gaps": not gapless},
        # graph-timed launches: p10 / median / p90 over the replays
        "per_launch_spread_us": {lbl: [round(a * 1e3, 3), round(t * 1e3, 3), round(b * 1e3, 3)]
                                 for (lbl, *_), t, (a, b) in zip(step, per_launch, per_launch_spread)},
        # after evicting L2 and the last-level cache: p10 / median / p90
        "per_launch_cold_us": {lbl: [round(float(np.percentile(c, q)) * 1e3, 3) for q in (10, 50, 90)]
                               for (lbl, *_), c in zip(step, cold)},
        "cold_timing": {"launches": KC, "evict_bytes": EVICT_BYTES},
        # every launch against the roof that bounds it (algorithmic work / duration)
        "per_launch_roofline": {lbl: (lambda r: f"{r['bound']} {r['frac']:.3f}")(
            roofline(kind, nums[li], t / 1e3)) for (lbl, li, kind, _), t in zip(step, per_launch)},
        "per_launch_roofline_cold": {lbl: (lambda r: f"{r['bound']} {r['frac']:.3f}")(
            roofline(kind, nums[li], t / 1e3)) for (lbl, li, kind, _), t in zip(step, cold_med)},
        # the weight transform (offline in the method): per-launch durations,
        # and the step with it included (eager, outside the timed region)
        "filter_transform_us": round(sum(filter_us), 3),
        "ms_per_step_with_filter_transform": round(full_ms, 6),
        "value_with_filter_transform": round(direct / (full_ms / 1e3) / 1e9, 1),
        "eager_ms_per_step": round(eager_ms, 6),
        "graph_ms_per_step": round(graph_ms, 6) if graph_ms is not None else None,
        "wall_ms_per_step": round((wall1 - wall0) * 1e3 / args.steps, 6),
        "copy_calibration_gbs": round(copy_gbs, 1),
        # what this chip sustains, beside the published peaks the roofline uses
        "measured_peaks": {"hbm_copy_gbs": round(copy_gbs, 1), "mfma_f32_tflops": round(mfma_tflops, 1),
                           "published_hbm_gbs": HBM_PEAK / 1e9, "published_mfma_f32_tflops": FP32_MFMA_PEAK / 1e12},
    }

    # CPU baseline: the fp64 oracle on this host, on a bounded sample (the first
    # layer, repeated until the time budget is spent); also checks the GPU output.
    if args.cpu_seconds > 0:
        from oracle import direct as odirect
        L0, g0 = w.first, gs[0]
        y_gpu = ys[0].detach().cpu().numpy()      # holds the last step's output (ReLU applied)
        if L0.nhwc:
            y_gpu = y_gpu.transpose(0, 3, 1, 2)
        reps_cpu, t_cpu, ref = 0, 0.0, None
        xin, pad_in = x, L0.pad
        if L0.axis:                    # 1-D layer: padding along the filtered axis only
            pw = [(0, 0)] * 4
            pw[3 if L0.axis == "w" else 2] = (L0.pad, L0.pad)
            xin, pad_in = np.pad(x, pw), 0
        while t_cpu < args.cpu_seconds and reps_cpu < 100000:
            t0 = time.perf_counter()
            ref = odirect.conv2d(xin, g0, pad_in)
            t_cpu += time.perf_counter() - t0
            reps_cpu += 1
        if L0.relu:
            ref = np.maximum(ref, 0.0)
        err = float(np.abs(y_gpu - ref).max() / max(np.abs(ref).max(), 1e-300))
        result["cpu_baseline"] = {
            "value": round(nums[0]["direct_flops"] * reps_cpu / t_cpu / 1e9, 3),
            "unit": "GFLOP/s", "cores": odirect.num_threads(), "kind": "oracle",
            "sample": f"layer 0 of {name} (whole layer, N={N}), {reps_cpu} run(s), {t_cpu:.1f} s"}
        result["max_rel_err_layer0"] = err
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
