#!/usr/bin/env python3
"""Benchmark of the N:M sparse INT8 GEMM on one MI355X.

Metric: dense-equivalent INT8 TOPS (2 m n k / t) of the sparse GEMMs of a ViT
workload, and their speedup over the dense INT8 MFMA GEMM of the same shapes.

One step = one pass over every linear of the workload: for each GEMM the
sparse kernel (nm_spmm on the packed weight) and the dense baseline
(nm_gemm_i8_dense on the same weight stored densely), interleaved.  Inputs
are resident in HBM before timing starts; packing is offline and untimed
(the paper times inference only, Sec. 6.1).  Every launch is bracketed by HIP
events on the stream it runs on; each step starts with a short device-side
sleep so the host has queued the whole step before the GPU reaches it, which
keeps host launch overhead out of the per-kernel times.

Prints one JSON line on stdout; human-readable tables go to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_12505_amd import nmspmm  # noqa: E402
from paper_2607_12505_amd import workloads as wl  # noqa: E402

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_INT8_TOPS = 5033.0        # dense INT8 MFMA: 256 CU x 2.4 GHz x 8192 op/clk
PEAK_SPARSE_TOPS = 10066.0     # structured-sparse INT8 (dense-equivalent)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pattern_name(g):
    return "dense" if g.N == g.M else f"{g.N}:{g.M}"


def algorithmic_bytes(g, out_i32, out_f16, sparse=True):
    """Bytes the GEMM must move at least once: X, the weight (compact packed
    form for sparse: N/M of the values plus ceil(log2 M) bits per kept value),
    the outputs and the scales."""
    b = g.m * g.k
    if sparse and g.N < g.M:
        bits = int(np.ceil(np.log2(g.M)))
        b += g.n * g.k * g.N // g.M + g.n * (g.k // g.M) * g.N * bits // 8
    else:
        b += g.n * g.k
    if out_i32:
        b += 4 * g.m * g.n
    if out_f16:
        b += 2 * g.m * g.n + 4 * g.n
    return b


class Prepared:
    """One GEMM of the workload with device buffers and ready-made ctypes
    arguments for both the sparse call and the dense baseline."""

    def __init__(self, cfg, g, x_dev_cache, x_host_cache, out_i32, out_f16, torch, use_dense_kernel):
        self.g = g
        X, W, scale = wl.inputs_for(cfg, g, x_host_cache)
        key = (g.m, g.k, g.layer, g.linear)
        if key not in x_dev_cache:
            x_dev_cache[key] = torch.from_numpy(X).cuda()
        self.X_host, self.W_host, self.scale_host = X, W, scale
        self.Xd = x_dev_cache[key]
        self.sparse_kernel = not use_dense_kernel
        self.Wd = torch.from_numpy(W).cuda()
        self.scale = torch.from_numpy(scale).cuda()
        self.Y = torch.empty((g.m, g.n), dtype=torch.int32, device="cuda") if out_i32 else None
        self.Yh = torch.empty((g.m, g.n), dtype=torch.int16, device="cuda") if out_f16 else None
        self.Yd = torch.empty((g.m, g.n), dtype=torch.int32, device="cuda") if out_i32 else None
        self.Yhd = torch.empty((g.m, g.n), dtype=torch.int16, device="cuda") if out_f16 else None
        out = (nmspmm.NM_OUT_I32 if out_i32 else 0) | (nmspmm.NM_OUT_F16 if out_f16 else 0)
        self.out_i32, self.out_f16 = out_i32, out_f16
        L = nmspmm.lib()
        ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        # dense baseline
        self.dplan = nmspmm.dense_plan(g.m, g.n, g.k, out)
        dws = nmspmm.workspace_size(self.dplan, g.m, g.n)
        self.dws = torch.zeros(max(dws, 16), dtype=torch.uint8, device="cuda")
        self.dense_args = (ptr(self.Xd), g.m, ptr(self.Wd), g.n, g.k, ptr(self.Yd), ptr(self.scale),
                           ptr(self.Yhd), ptr(self.dws), self.dws.numel(), stream, ctypes.byref(self.dplan))
        self.dense_fn = L.nm_gemm_i8_dense_ex
        if self.sparse_kernel:
            self.packed = nmspmm.compress(W, g.N, g.M)
            self.dw = nmspmm.DeviceWeight.from_packed(self.packed)
            self.splan = nmspmm.spmm_plan(self.packed.desc, g.m, out)
            sws = nmspmm.workspace_size(self.splan, g.m, g.n)
            self.sws = torch.zeros(max(sws, 16), dtype=torch.uint8, device="cuda")
            self.sparse_args = (ptr(self.Xd), g.m, ptr(self.dw.vals), ptr(self.dw.meta),
                                ctypes.byref(self.packed.desc), ptr(self.Y), ptr(self.scale), ptr(self.Yh),
                                ptr(self.sws), self.sws.numel(), stream, ctypes.byref(self.splan))
            self.sparse_fn = L.nm_spmm_ex
        else:
            # a dense layer inside a layer-wise chain runs the dense kernel on both sides
            self.splan = self.dplan
            self.sparse_args = (ptr(self.Xd), g.m, ptr(self.Wd), g.n, g.k, ptr(self.Y), ptr(self.scale),
                                ptr(self.Yh), ptr(self.dws), self.dws.numel(), stream, ctypes.byref(self.dplan))
            self.sparse_fn = L.nm_gemm_i8_dense_ex

    def kernel_name(self, plan):
        kind = {1: "sp42", 2: "sp42x2", 3: "dense"}[plan.kind]
        return f"{kind}/t{plan.tile_n}x{plan.tile_m}"

    def run_sparse(self):
        st = self.sparse_fn(*self.sparse_args)
        if st:
            raise nmspmm.NmError(st, f"sparse {self.g.name}")

    def run_dense(self):
        st = self.dense_fn(*self.dense_args)
        if st:
            raise nmspmm.NmError(st, f"dense {self.g.name}")


def time_steps(preps, steps, torch, sleep_cycles):
    """Runs `steps` steps; returns per-launch times [steps, gemms, 2] in ms."""
    E = torch.cuda.Event
    ev = [[(E(enable_timing=True), E(enable_timing=True), E(enable_timing=True)) for _ in preps]
          for _ in range(steps)]
    for s in range(steps):
        if sleep_cycles:
            torch.cuda._sleep(sleep_cycles)
        for i, p in enumerate(preps):
            e0, e1, e2 = ev[s][i]
            e0.record()
            p.run_sparse()
            e1.record()
            p.run_dense()
            e2.record()
    torch.cuda.synchronize()
    t = np.zeros((steps, len(preps), 2))
    for s in range(steps):
        for i in range(len(preps)):
            e0, e1, e2 = ev[s][i]
            t[s, i, 0] = e0.elapsed_time(e1)
            t[s, i, 1] = e1.elapsed_time(e2)
    return t


def cpu_baseline(preps, budget_s, check):
    """The oracle (plain C, all host threads) on the first rows of every GEMM
    of the workload; the row fraction is sized to about budget_s seconds."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    # calibrate on a small slice of the largest GEMM
    big = max(preps, key=lambda p: p.g.m * p.g.n * p.g.k)
    rows = max(1, min(big.g.m, 64))
    t0 = time.perf_counter()
    oracle.matmul_i8(big.X_host[:rows], big.W_host, nthreads=threads)
    rate = 2.0 * rows * big.g.n * big.g.k / max(time.perf_counter() - t0, 1e-6)
    total = sum(2.0 * p.g.m * p.g.n * p.g.k for p in preps)
    frac = min(1.0, budget_s * rate / total)
    ops = 0.0
    mism = 0
    t0 = time.perf_counter()
    for p in preps:
        r = max(1, int(round(p.g.m * frac)))
        Yc = oracle.matmul_i8(p.X_host[:r], p.W_host, nthreads=threads)
        ops += 2.0 * r * p.g.n * p.g.k
        if check and p.Y is not None:
            mism += int((p.Y[:r].cpu().numpy() != Yc).sum())
    dt = time.perf_counter() - t0
    return {
        "value": ops / dt / 1e12,
        "unit": "TOPS (dense-equivalent INT8)",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {frac * 100:.2f}% of the rows of each of the {len(preps)} GEMMs "
                  f"({ops / 1e9:.1f} dense-eq GOP in {dt:.1f} s)",
    }, mism


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=1, help="0..4 (default 1: DeiT-Small linears, batch 64)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic", type=str, default=None,
                    help="JSON file with measured HBM bytes per launch of the dominant kernel")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the method is a "
              "single-GPU kernel; see the sharding notes in DESIGN.md)", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    nmspmm.lib()
    torch.cuda.set_device(0)

    work = wl.workload(args.config)
    out_i32, out_f16 = work.out_int32, work.out_f16
    log(f"workload {work.name}: {len(work.gemms)} GEMMs, outputs "
        f"{'int32' if out_i32 else ''}{'+fp16' if out_f16 else ''}")
    t0 = time.perf_counter()
    xd, xh = {}, {}
    preps = [Prepared(args.config, g, xd, xh, out_i32, out_f16, torch, use_dense_kernel=(g.N == g.M))
             for g in work.gemms]
    torch.cuda.synchronize()
    log(f"inputs generated, packed and uploaded in {time.perf_counter() - t0:.1f} s")

    # sleep long enough for the host to enqueue one step ahead of the GPU
    sleep_cycles = int(2.4e9 * 25e-6 * len(preps) * 2)
    time_steps(preps, max(1, args.warmup), torch, sleep_cycles)

    torch.cuda.synchronize()
    w0 = time.perf_counter()
    t = time_steps(preps, args.steps, torch, sleep_cycles)
    wall = time.perf_counter() - w0
    ms_per_step = wall * 1e3 / args.steps

    # per GEMM: mean over steps (the paper averages repeated runs, Sec. 5.1)
    ts = t[:, :, 0].mean(axis=0)
    td = t[:, :, 1].mean(axis=0)
    ops = np.array([p.g.dense_eq_ops for p in preps], np.float64)
    sparse_sel = np.array([p.sparse_kernel for p in preps])
    value = ops[sparse_sel].sum() / (ts[sparse_sel].sum() * 1e-3) / 1e12
    dense_tops = ops.sum() / (td.sum() * 1e-3) / 1e12
    speedup = td[sparse_sel].sum() / ts[sparse_sel].sum()

    per_pattern = {}
    for pat in sorted({pattern_name(p.g) for p in preps}):
        sel = np.array([pattern_name(p.g) == pat for p in preps])
        per_pattern[pat] = {
            "tops": round(float(ops[sel].sum() / (ts[sel].sum() * 1e-3) / 1e12), 1),
            "speedup_vs_dense": round(float(td[sel].sum() / ts[sel].sum()), 3),
        }

    # dominant kernel: the (kind, tile) instantiation with the most sparse time per step
    groups = {}
    for i, p in enumerate(preps):
        if not p.sparse_kernel:
            continue
        name = p.kernel_name(p.splan)
        gr = groups.setdefault(name, {"time_ms": 0.0, "bytes": 0, "ops": 0.0, "launches": 0, "split": set()})
        gr["time_ms"] += ts[i]
        gr["bytes"] += algorithmic_bytes(p.g, out_i32, out_f16)
        gr["ops"] += ops[i]
        gr["launches"] += 1
        gr["split"].add(p.splan.split_k)
    dom_name = max(groups, key=lambda k: groups[k]["time_ms"])
    dom = groups[dom_name]
    avg_ms = dom["time_ms"] / dom["launches"]
    achieved = dom["bytes"] / dom["launches"] / (avg_ms * 1e-3) / 1e9
    traffic = None
    if args.traffic and os.path.exists(args.traffic):
        with open(args.traffic) as f:
            tr = json.load(f)
        if tr.get("kernel") == dom_name and tr.get("workload") == work.name:
            traffic = tr.get("bytes_per_launch")
    roofline = {
        "bound": "hbm",
        "achieved": round(achieved, 1),
        "peak": PEAK_HBM_GBS,
        "unit": "GB/s",
        "frac": round(achieved / PEAK_HBM_GBS, 4),
        "traffic": traffic,
        "kernel": dom_name,
        "launches_per_step": dom["launches"],
        "avg_launch_us": round(avg_ms * 1e3, 2),
        "algorithmic_bytes_per_launch": int(dom["bytes"] / dom["launches"]),
    }

    log(f"\n{'gemm':<22}{'m':>7}{'k':>6}{'n':>6}  {'plan':<18}{'sparse us':>10}{'dense us':>10}"
        f"{'TOPS':>8}{'dTOPS':>8}{'spd':>7}{'GB/s':>8}")
    for i, p in enumerate(preps):
        g = p.g
        b = algorithmic_bytes(g, out_i32, out_f16, sparse=p.sparse_kernel)
        log(f"{g.name:<22}{g.m:>7}{g.k:>6}{g.n:>6}  {p.kernel_name(p.splan) + '/s' + str(p.splan.split_k):<18}"
            f"{ts[i] * 1e3:>10.1f}{td[i] * 1e3:>10.1f}{ops[i] / ts[i] / 1e9:>8.0f}{ops[i] / td[i] / 1e9:>8.0f}"
            f"{td[i] / ts[i]:>7.2f}{b / ts[i] / 1e6:>8.0f}")
    log(f"\nsparse {value:.1f} TOPS dense-eq, dense {dense_tops:.1f} TOPS, speedup {speedup:.3f}; "
        f"dominant kernel {dom_name}: {achieved:.0f} GB/s ({achieved / PEAK_HBM_GBS * 100:.1f}% of HBM peak)")

    line = {
        "metric": "dense-equivalent INT8 TOPS and speedup vs dense INT8 MFMA GEMM, per N:M ratio",
        "value": round(float(value), 2),
        "unit": "TOPS (dense-equivalent INT8)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded: X uniform int8, W N(0,0.02) pruned top-N per window, per-row int8)",
        "config": {
            "workload": work.name,
            "gemms": len(preps),
            "m": sorted({p.g.m for p in preps}),
            "patterns": sorted({pattern_name(p.g) for p in preps}),
            "outputs": ("int32" if out_i32 else "") + ("+fp16" if out_f16 else ""),
        },
        "speedup_vs_dense": round(float(speedup), 3),
        "dense_tops": round(float(dense_tops), 2),
        "frac_of_int8_peak": round(float(value / PEAK_INT8_TOPS), 4),
        "per_pattern": per_pattern,
        "sparse_ms_per_step": round(float(ts[sparse_sel].sum()), 4),
        "dense_ms_per_step": round(float(td.sum()), 4),
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        cb, mism = cpu_baseline(preps, args.cpu_budget, check=True)
        line["cpu_baseline"] = cb
        line["parity_sampled_rows_mismatches"] = mism
        log(f"cpu oracle: {cb['value'] * 1e3:.2f} GOPS on {cb['cores']} threads; "
            f"GPU vs oracle on those rows: {mism} mismatches")
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
