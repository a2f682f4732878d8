#!/usr/bin/env python3
"""Benchmark of the Winograd hot path on one MI355X.

One step = one pass of the whole path over one batch: the weight transform and
the convolution (input transform -> T GEMMs -> output transform) of every 3x3
layer in the workload (plus the 2x2 pools of a stack).  Prints one JSON line.

Metric: effective GFLOP/s = direct-convolution FLOPs (2*N*K*C*9*Ho*Wo per layer)
divided by the step time.  Also reported: the roofline position of the
dominant kernel (its average duration from HIP events on the launch stream), and
the fp64 CPU oracle timed on this host on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK = 8.0e12          # B/s, MI355X HBM3E
FP32_MFMA_PEAK = 157.3e12  # FLOP/s, MI355X dense fp32 matrix


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def layer_numbers(N, L):
    """Sizes and algorithmic work of one layer (m x m tiles, alpha = m+2)."""
    Ho, Wo = L.H + 2 * L.pad - 2, L.W + 2 * L.pad - 2
    th, tw = -(-Ho // L.m), -(-Wo // L.m)
    P = N * th * tw
    T = (L.m + 2) ** 2
    Cp, Kp = -(-L.C // 4) * 4, -(-L.K // 16) * 16
    f = dict(Ho=Ho, Wo=Wo, P=P, T=T)
    f["direct_flops"] = 2 * N * L.K * L.C * 9 * Ho * Wo
    f["gemm_flops"] = 2 * T * P * L.C * L.K
    x_b, y_b, u_b = 4 * N * L.C * L.H * L.W, 4 * N * L.K * Ho * Wo, 4 * T * Cp * Kp
    v_b, m_b = 4 * T * P * L.C, 4 * T * P * L.K
    # minimum HBM bytes per kernel (what the method must move, padding excluded)
    f["bytes"] = {
        "filter": 4 * L.K * L.C * 9 + u_b,
        "fused": x_b + u_b + y_b,
        "input": x_b + v_b,
        "gemm": v_b + u_b + m_b,
        "output": m_b + y_b,
        "maxpool": y_b + y_b // 4,
    }
    f["flops"] = {"fused": f["gemm_flops"], "gemm": f["gemm_flops"]}
    return f


def roofline(kind, nums, seconds):
    b = nums["bytes"].get(kind, 0)
    fl = nums["flops"].get(kind, 0)
    t_hbm = b / HBM_PEAK
    t_mfma = fl / FP32_MFMA_PEAK
    if t_mfma >= t_hbm and fl > 0:
        ach = fl / seconds / 1e12
        return {"bound": "mfma", "achieved": round(ach, 3), "peak": FP32_MFMA_PEAK / 1e12,
                "unit": "TFLOP/s", "frac": round(ach / (FP32_MFMA_PEAK / 1e12), 4), "traffic": None}
    ach = b / seconds / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": round(ach / (HBM_PEAK / 1e9), 4), "traffic": None}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--algo", choices=["auto", "fused", "staged"], default="auto")
    ap.add_argument("--flags", type=lambda s: int(s, 0), default=None,
                    help="explicit wino_conv2d flags (overrides --algo)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU time budget of the oracle baseline (0 disables it)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
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

    x, gs = wl.generate(w)
    dev = torch.device("cuda:0")
    hx = torch.from_numpy(x).to(dev)
    hg = [torch.from_numpy(g).to(dev) for g in gs]
    nums = [layer_numbers(N, L) for L in w.layers]

    # Device buffers, all allocated before timing.
    Us, ys, pools, wss, Vs, Ms = [], [], [], [], [], []
    H, W = w.first.H, w.first.W
    for L, f in zip(w.layers, nums):
        assert (L.H, L.W) == (H, W)
        Us.append(torch.empty(B.wino_filter_bytes(L.C, L.K, L.m) // 4, dtype=torch.float32, device=dev))
        ys.append(torch.empty((N, L.K, f["Ho"], f["Wo"]), dtype=torch.float32, device=dev))
        wsb = B.wino_workspace_bytes(N, L.C, L.H, L.W, L.K, L.pad, L.m, flags)
        wss.append((torch.empty(max(wsb // 4, 1), dtype=torch.float32, device=dev), wsb))
        if staged:
            Vs.append(torch.empty(B.wino_input_tf_bytes(N, L.C, L.H, L.W, L.pad, L.m) // 4,
                                  dtype=torch.float32, device=dev))
            Ms.append(torch.empty(B.wino_gemm_out_bytes(N, L.K, L.H, L.W, L.pad, L.m) // 4,
                                  dtype=torch.float32, device=dev))
        H, W = f["Ho"], f["Wo"]
        if L.pool:
            pools.append(torch.empty((N, L.K, H // 2, W // 2), dtype=torch.float32, device=dev))
            H, W = H // 2, W // 2
        else:
            pools.append(None)

    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    def launches():
        """The step as a list of (label, layer index, kind, thunk)."""
        out = []
        a = hx
        for i, L in enumerate(w.layers):
            relu = B.WINO_FLAG_RELU if L.relu else 0
            out.append((f"L{i}.filter", i, "filter",
                        (lambda i=i, L=L: B.wino_filter_transform(hg[i], Us[i], L.C, L.K, L.m, sp))))
            if staged:
                out.append((f"L{i}.input", i, "input", (lambda i=i, L=L, a=a: B.wino_input_transform(
                    a, Vs[i], N, L.C, L.H, L.W, L.pad, L.m, sp))))
                out.append((f"L{i}.gemm", i, "gemm", (lambda i=i, L=L: B.wino_batched_gemm(
                    Us[i], Vs[i], Ms[i], N, L.C, L.H, L.W, L.K, L.pad, L.m, sp))))
                out.append((f"L{i}.output", i, "output", (lambda i=i, L=L, relu=relu: B.wino_output_transform(
                    Ms[i], ys[i], N, L.K, L.H, L.W, L.pad, L.m, relu, sp))))
            else:
                ws, wsb = wss[i]
                out.append((f"L{i}.conv", i, "fused", (lambda i=i, L=L, a=a, relu=relu, ws=ws, wsb=wsb:
                                                       B.wino_conv2d(a, Us[i], ys[i], N, L.C, L.H, L.W, L.K,
                                                                     L.pad, L.m, flags | relu,
                                                                     ws if wsb else None, wsb, sp))))
            a = ys[i]
            if L.pool:
                out.append((f"L{i}.pool", i, "maxpool", (lambda i=i, L=L, a=a: B.wino_maxpool2x2(
                    a, pools[i], N, L.K, nums[i]["Ho"], nums[i]["Wo"], sp))))
                a = pools[i]
        return out

    step = launches()

    def run_step():
        for label, _, _, fn in step:
            st = fn()
            if st != 0:
                raise RuntimeError(f"{label}: {B.wino_status_string(st)}")

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    # Timed region: exactly K steps, synchronised on both sides.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        run_step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall1 = time.perf_counter()
    ms_step = e0.elapsed_time(e1) / args.steps

    # Per-kernel durations: the same K steps again with an event pair around
    # every launch, on the launch stream.
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in step]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        for j, (label, _, _, fn) in enumerate(step):
            evs[s][j][0].record(stream)
            fn()
            evs[s][j][1].record(stream)
    torch.cuda.synchronize()
    per_launch = [float(np.mean([evs[s][j][0].elapsed_time(evs[s][j][1]) for s in range(args.steps)]))
                  for j in range(len(step))]
    dom = int(np.argmax(per_launch))
    dlabel, dlayer, dkind, _ = step[dom]
    dsec = per_launch[dom] / 1e3
    roof = roofline(dkind, nums[dlayer], dsec)
    roof["kernel"] = dlabel
    roof["avg_us"] = round(per_launch[dom] * 1e3, 3)

    direct = sum(f["direct_flops"] for f in nums)
    value = direct / (ms_step / 1e3) / 1e9

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
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "N": N, "layers": len(w.layers),
                   "C": w.first.C, "K": w.first.K, "H": w.first.H, "W": w.first.W,
                   "m": w.first.m, "pad": w.first.pad, "flags": hex(flags), "parallelism": "none"},
        "roofline": roof,
        "per_launch_us": {lbl: round(t * 1e3, 3) for (lbl, *_), t in zip(step, per_launch)},
        "wall_ms_per_step": round((wall1 - wall0) * 1e3 / args.steps, 6),
    }

    # CPU baseline: the fp64 oracle on this host, on a bounded sample (the first
    # layer, repeated until the time budget is spent); also checks the GPU output.
    if args.cpu_seconds > 0:
        from oracle import direct as odirect
        L0, g0 = w.first, gs[0]
        y_gpu = ys[0].detach().cpu().numpy()      # holds the last step's output (ReLU applied)
        reps, t_cpu, ref = 0, 0.0, None
        while t_cpu < args.cpu_seconds and reps < 1000:
            t0 = time.perf_counter()
            ref = odirect.conv2d(x, g0, L0.pad)
            t_cpu += time.perf_counter() - t0
            reps += 1
        if L0.relu:
            ref = np.maximum(ref, 0.0)
        err = float(np.abs(y_gpu - ref).max() / max(np.abs(ref).max(), 1e-300))
        result["cpu_baseline"] = {
            "value": round(nums[0]["direct_flops"] * reps / t_cpu / 1e9, 3),
            "unit": "GFLOP/s", "cores": odirect.num_threads(), "kind": "oracle",
            "sample": f"layer 0 of {name} (whole layer, N={N}), {reps} run(s), {t_cpu:.1f} s"}
        result["max_rel_err_layer0"] = err
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
