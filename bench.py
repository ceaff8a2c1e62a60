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
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_12505_amd import nmprobe, nmspmm  # noqa: E402
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
        return nmspmm.plan_kernel_name(plan)

    def run_sparse(self):
        st = self.sparse_fn(*self.sparse_args)
        if st:
            raise nmspmm.NmError(st, f"sparse {self.g.name}")

    def run_dense(self):
        st = self.dense_fn(*self.dense_args)
        if st:
            raise nmspmm.NmError(st, f"dense {self.g.name}")


def launch_groups(preps):
    """Timed launch groups of a step: the sparse-side launches of one kernel
    instantiation, then likewise for the dense baseline.  Events bracket whole
    groups of back-to-back launches, so no event sits between two kernels of
    a group."""
    groups = {}
    for i, p in enumerate(preps):
        groups.setdefault(("sparse", p.kernel_name(p.splan)), []).append(i)
    for i, p in enumerate(preps):
        groups.setdefault(("dense", p.kernel_name(p.dplan)), []).append(i)
    return list(groups.items())


def time_steps(preps, groups, steps, torch, sleep_cycles):
    """Runs `steps` steps; returns group times [steps, groups] in ms."""
    E = torch.cuda.Event
    ev = [[E(enable_timing=True) for _ in range(len(groups) + 1)] for _ in range(steps)]
    for s in range(steps):
        if sleep_cycles:
            torch.cuda._sleep(sleep_cycles)
        ev[s][0].record()
        for gi, ((side, _), idx) in enumerate(groups):
            for i in idx:
                if side == "sparse":
                    preps[i].run_sparse()
                else:
                    preps[i].run_dense()
            ev[s][gi + 1].record()
    torch.cuda.synchronize()
    t = np.zeros((steps, len(groups)))
    for s in range(steps):
        for gi in range(len(groups)):
            t[s, gi] = ev[s][gi].elapsed_time(ev[s][gi + 1])
    return t


def graph_steps(preps, groups, steps, torch, sleep_cycles):
    """The step's launches captured once per side (sparse, dense) in a HIP
    graph, in the same group order, and replayed `steps` times behind the same
    device sleep; returns the mean sparse and dense milliseconds per step.
    The outputs are rewritten by every replay, so the sampled-row parity check
    that follows sees the graphs' results."""
    side = torch.cuda.Stream()
    h = ctypes.c_void_p(side.cuda_stream)

    def on_side(args):  # the stream is argument 10 of both entry points
        a = list(args)
        a[10] = h
        return tuple(a)
    calls = {"sparse": [], "dense": []}
    for (kind, _), idx in groups:
        for i in idx:
            p = preps[i]
            calls[kind].append((p.sparse_fn, on_side(p.sparse_args)) if kind == "sparse"
                               else (p.dense_fn, on_side(p.dense_args)))

    def run(kind):
        for fn, a in calls[kind]:
            st = fn(*a)
            if st:
                raise nmspmm.NmError(st, f"graph step ({kind})")
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run("sparse")
        run("dense")
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = {}
    for kind in ("sparse", "dense"):
        graphs[kind] = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graphs[kind], stream=side):
            run(kind)
    torch.cuda.synchronize()
    E = torch.cuda.Event
    ev = [[E(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for s in range(steps):
        if sleep_cycles:
            torch.cuda._sleep(sleep_cycles)
        ev[s][0].record()
        graphs["sparse"].replay()
        ev[s][1].record()
        graphs["dense"].replay()
        ev[s][2].record()
    torch.cuda.synchronize()
    sp = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    dn = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    return sp, dn


def time_each(preps, torch, reps=5):
    """Untimed detail pass: mean time of each GEMM, sparse and dense, each
    over `reps` back-to-back launches (for the per-GEMM table only)."""
    E = torch.cuda.Event
    out = np.zeros((len(preps), 2))
    for i, p in enumerate(preps):
        for side, fn in ((0, p.run_sparse), (1, p.run_dense)):
            fn()
            torch.cuda.synchronize()
            torch.cuda._sleep(int(2.4e9 * 20e-6 * reps))
            e0, e1 = E(enable_timing=True), E(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            out[i, side] = e0.elapsed_time(e1) / reps
    return out


def store_only_time(preps, idx, torch, reps=10):
    """Mean time per launch of the GEMMs `idx` with their reduction skipped
    (nm_probe_store_only: the same plans, outputs and epilogue stores, no
    loads or matrix work), timed like a launch group of the step; None if a
    plan's layout has no such mode.  The real results are written back
    afterwards."""
    L = nmprobe.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    calls = []
    for i in idx:
        p = preps[i]
        o = nmspmm.NmOutputs(p.Y.data_ptr() if p.Y is not None else None,
                             p.Yh.data_ptr() if p.Yh is not None else None,
                             p.scale.data_ptr(), None, None)
        calls.append((ctypes.byref(p.splan), p.g.m, p.g.n, o))
    for plan, m, n, o in calls:
        if L.nm_probe_store_only(plan, m, n, ctypes.byref(o), stream) != nmspmm.NM_OK:
            return None
    E = torch.cuda.Event
    ev = [(E(enable_timing=True), E(enable_timing=True)) for _ in range(reps)]
    for e0, e1 in ev:
        torch.cuda._sleep(int(2.4e9 * 25e-6 * len(calls)))
        e0.record()
        for plan, m, n, o in calls:
            L.nm_probe_store_only(plan, m, n, ctypes.byref(o), stream)
        e1.record()
    torch.cuda.synchronize()
    for i in idx:  # the real results again, for the parity check that follows
        preps[i].run_sparse()
    torch.cuda.synchronize()
    return float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev])) / len(calls)


def chain_times(preps, torch, reps, sleep_cycles):
    """A chain workload in network order: one event pair around all its
    launches, back to back on one stream (the sparse chain, then the all-dense
    chain), behind the step's device sleep; mean milliseconds per chain."""
    E = torch.cuda.Event
    ev = [[E(enable_timing=True) for _ in range(4)] for _ in range(reps)]
    for r in range(reps):
        for side in (0, 1):
            torch.cuda._sleep(sleep_cycles)
            ev[r][2 * side].record()
            for p in preps:
                p.run_dense() if side else p.run_sparse()
            ev[r][2 * side + 1].record()
    torch.cuda.synchronize()
    sp = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    dn = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
    return sp, dn


def time_keyed_in_steps(preps, key, torch, reps):
    """Untimed detail pass in the step's own cache state: `reps` whole steps in
    which the GEMMs are ordered by `key(prep)` (sparse calls of each key, then
    the dense calls of each key) with an event at every key boundary only, so
    no event separates two GEMMs of one key; returns {key: (sparse ms, dense
    ms)} per step.  Each step starts behind a device sleep long enough for the
    host to queue it."""
    E = torch.cuda.Event
    keys = sorted({key(p) for p in preps})
    members = {k: [p for p in preps if key(p) == k] for k in keys}
    sleep_cycles = int(2.4e9 * 25e-6 * 2 * len(preps))
    ev = [[E(enable_timing=True) for _ in range(2 * len(keys) + 1)] for _ in range(reps)]
    for r in range(reps):
        torch.cuda._sleep(sleep_cycles)
        ev[r][0].record()
        for side in (0, 1):
            for j, k in enumerate(keys):
                for p in members[k]:
                    p.run_dense() if side else p.run_sparse()
                ev[r][side * len(keys) + j + 1].record()
    torch.cuda.synchronize()
    out = {}
    for j, k in enumerate(keys):
        sp = np.mean([ev[r][j].elapsed_time(ev[r][j + 1]) for r in range(reps)])
        dn = np.mean([ev[r][len(keys) + j].elapsed_time(ev[r][len(keys) + j + 1]) for r in range(reps)])
        out[k] = (float(sp), float(dn))
    return out


def secondary_workload(cfg, steps, warmup, torch):
    """Speedup over the dense baseline per (token count, N:M) on another
    workload (same protocol as the main measurement, fewer steps); reported
    beside the main line, never folded into its value."""
    work = wl.workload(cfg)
    xd, xh = {}, {}
    preps = [Prepared(cfg, g, xd, xh, work.out_int32, work.out_f16, torch, use_dense_kernel=(g.N == g.M))
             for g in work.gemms]
    torch.cuda.synchronize()
    sleep_cycles = int(2.4e9 * 25e-6 * len(preps) * 2)
    groups = launch_groups(preps)
    time_steps(preps, groups, max(1, warmup), torch, sleep_cycles)
    keyfn = lambda p: (p.g.m, pattern_name(p.g))
    times = time_keyed_in_steps(preps, keyfn, torch, 3 * steps)
    out = {}
    for key, (ts, td) in times.items():
        ops = sum(p.g.dense_eq_ops for p in preps if keyfn(p) == key)
        out[f"m={key[0]} {key[1]}"] = {"tops": round(ops / (ts * 1e-3) / 1e12, 1),
                                        "speedup_vs_dense": round(float(td / ts), 3)}
    del preps
    torch.cuda.empty_cache()
    return {"workload": work.name, "outputs": "int32", "per_batch_pattern": out}


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
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    from oracle import build as oracle_build
    return {
        "value": ops / dt / 1e12,
        "unit": "TOPS (dense-equivalent INT8)",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": model,
        "compiler": "gcc " + " ".join(oracle_build.CFLAGS),
        "sample": f"first {frac * 100:.2f}% of the rows of each of the {len(preps)} GEMMs "
                  f"({ops / 1e9:.1f} dense-eq GOP in {dt:.1f} s)",
    }, mism


def sweep_summary(rows):
    """Table-1 figures of a set of sweep rows: the planner's Top-1 hit rate, its
    average and worst time normalised to the sweep optimum, and the gain over a
    fixed split_k = 1 with the planner's tile."""
    if not rows:
        return None
    norm = np.array([r["t_best_us"] / r["t_planned_us"] for r in rows])
    fixed = np.array([r["t_fixed_split1_us"] / r["t_planned_us"] for r in rows if r["t_fixed_split1_us"]])
    fixed_tile = np.array([r["times"]["16/1"] / r["t_planned_us"] for r in rows if r["times"].get("16/1")])
    return {
        "cases": len(rows),
        "top1_hit_rate": round(float(np.mean([r["planned"] == r["best"] for r in rows])), 3),
        "avg_norm_perf": round(float(norm.mean()), 3),
        "worst_norm_perf": round(float(norm.min()), 3),
        "gain_over_fixed_split1": round(float(fixed.mean()), 3) if len(fixed) else None,
        # against one fixed plan for every shape (128 x 128, no split)
        "gain_over_fixed_128x128": round(float(fixed_tile.mean()), 3) if len(fixed_tile) else None,
    }


GRID_PATTERNS = (((2, 4), 50), ((4, 8), 50), ((1, 4), 75), ((2, 8), 75), ((1, 8), 87.5))


def paper_grid_workload():
    """The paper's kernel benchmark grid (Sec. 6.1) as a sweep workload: m in
    {64, 128, 256, 512}, n and k in {128, 256, 512, 1024}, the five patterns of
    50 / 75 / 87.5 % sparsity, int32 output."""
    sizes = (128, 256, 512, 1024)
    gemms = tuple(wl.Gemm(f"m{m} n{n} k{k} {N}:{M}", m, k, n, N, M)
                  for m in (64, 128, 256, 512) for n in sizes for k in sizes for (N, M), _ in GRID_PATTERNS)
    return wl.Workload(-1, "paper_kernel_grid", gemms)


def sweep(configs, torch, reps, out_path):
    """Planner evaluation in the manner of the paper's Table 1: for every
    distinct (shape, N:M) of the workloads, time every (tile, split_k)
    candidate; the fastest is the sweep optimum.  Reports the planner's Top-1
    hit rate, its average and worst performance normalised to the optimum, and
    the gain over a fixed split_k = 1 setting (same tile)."""
    E = torch.cuda.Event
    rows = []
    seen = set()
    for cfg in configs:
        work = paper_grid_workload() if cfg == "grid" else wl.workload(cfg)
        out = (nmspmm.NM_OUT_I32 if work.out_int32 else 0) | (nmspmm.NM_OUT_F16 if work.out_f16 else 0)
        cases = []
        for g in work.gemms:
            cases.append(g)
            if g.N < g.M:
                # the dense baseline of the same shape, whose plan is the
                # denominator of every speedup
                base = " ".join(t for t in g.name.split() if ":" not in t)
                cases.append(dataclasses.replace(g, name="dense " + base, N=8, M=8))
        for g in cases:
            key = (g.m, g.k, g.n, g.N == g.M or (g.N, g.M), out)
            if key in seen:
                continue
            seen.add(key)
            if cfg == "grid":
                rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([6, g.m, g.n, g.k, g.N, g.M])))
                X = wl.gen_x(g.m, g.k, rng)
                W, scale = wl.gen_w(g.n, g.k, g.N, g.M, rng)
            else:
                X, W, scale = wl.inputs_for(cfg, g)
            Xd = torch.from_numpy(X).cuda()
            sd = torch.from_numpy(scale).cuda()
            sparse = g.N < g.M
            if sparse:
                dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, g.N, g.M))
                planned = nmspmm.spmm_plan(dw.desc, g.m, out)
            else:
                Wd = torch.from_numpy(W).cuda()
                planned = nmspmm.dense_plan(g.m, g.n, g.k, out)
            # rotate the outputs over at least two buffers and 512 MB in all
            # (twice the last-level cache), as a network's consecutive layers
            # write fresh buffers
            out_bytes = g.m * g.n * ((4 if out & 1 else 0) + (2 if out & 2 else 0))
            nsets = int(min(64, max(2, -(-512e6 // out_bytes))))
            Ys = [torch.empty((g.m, g.n), dtype=torch.int32, device="cuda") if out & 1 else None for _ in range(nsets)]
            Yhs = [torch.empty((g.m, g.n), dtype=torch.int16, device="cuda") if out & 2 else None for _ in range(nsets)]
            ws = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda")
            times = {}
            cursor = 0  # the next output buffer in the rotation
            # two passes over the candidates, the second in reverse order,
            # keeping each one's faster mean: a candidate slowed once by a
            # transient (clock or power state left by the kernels before it)
            # is not mistaken for a slow schedule
            order = list(range(nmspmm.num_tiles()))
            for tile in order + order[::-1]:
                tn_, tm_ = nmspmm.tile_info(tile)
                tiles = -(-g.n // tn_) * -(-g.m // tm_)
                for split in (1, 2, 4, 8):
                    if split > 1 and tiles >= 256 and (tile, split) != (planned.tile, planned.split_k):
                        continue  # split-K only where the tiles alone leave compute units idle
                    plan = nmspmm.make_plan(planned.kind, tile, split)
                    try:
                        if nmspmm.workspace_size(plan, g.m, g.n) > ws.numel():
                            continue
                        def run(i, plan=plan):
                            if sparse:
                                nmspmm.spmm(Xd, dw, Y=Ys[i], scale=sd, Yh=Yhs[i], plan=plan, ws=ws)
                            else:
                                nmspmm.gemm_i8_dense(Xd, Wd, Y=Ys[i], scale=sd, Yh=Yhs[i], plan=plan, ws=ws)
                        run(0)
                    except nmspmm.NmError:
                        continue
                    torch.cuda.synchronize()
                    # queue the launches behind a 1 ms spin, which also lets
                    # the clock recover from the previous candidate
                    torch.cuda._sleep(int(2.4e9 * 100e-6 * reps))
                    e0, e1 = E(enable_timing=True), E(enable_timing=True)
                    e0.record()
                    for r in range(reps):
                        run(cursor % nsets)
                        cursor += 1
                    e1.record()
                    torch.cuda.synchronize()
                    t_us = e0.elapsed_time(e1) / reps * 1e3
                    times[(tile, split)] = min(t_us, times.get((tile, split), t_us))
            best = min(times, key=times.get)
            chosen = (planned.tile, planned.split_k)
            t_plan = times.get(chosen)
            t_fixed = times.get((planned.tile, 1))
            rows.append({
                "cfg": cfg, "gemm": g.name, "m": g.m, "k": g.k, "n": g.n, "pattern": pattern_name(g),
                "planned": list(chosen), "best": list(best), "t_planned_us": t_plan, "t_best_us": times[best],
                "t_fixed_split1_us": t_fixed, "times": {f"{t}/{s}": v for (t, s), v in times.items()},
            })
            log(f"cfg{cfg} {g.name:<20} m={g.m:<6} k={g.k:<5} n={g.n:<5} planned t{chosen[0]}/s{chosen[1]} "
                f"{t_plan:7.1f} us  best t{best[0]}/s{best[1]} {times[best]:7.1f} us  "
                f"norm {times[best] / t_plan:.3f}")
    summary = sweep_summary([r for r in rows if r["pattern"] != "dense" and r["cfg"] != "grid"])
    dense_summary = sweep_summary([r for r in rows if r["pattern"] == "dense" and r["cfg"] != "grid"])
    # the paper's Table 1 rows: the kernel grid per sparsity (and its dense baseline)
    spars = {f"{N}:{M}": sp for (N, M), sp in GRID_PATTERNS}
    grid_summary = None
    if "grid" in configs:
        grid_summary = {str(sp): sweep_summary([r for r in rows if r["cfg"] == "grid" and
                                                spars.get(r["pattern"]) == sp]) for sp in (50, 75, 87.5)}
        grid_summary["dense"] = sweep_summary([r for r in rows if r["cfg"] == "grid" and r["pattern"] == "dense"])
    log(json.dumps({"sparse": summary, "dense": dense_summary, "grid": grid_summary}))
    if out_path:
        with open(out_path, "w") as f:
            json.dump({"summary": summary, "dense_summary": dense_summary, "grid_summary": grid_summary,
                       "rows": rows}, f, indent=1)
    return summary


def predictor_experiment(torch, n_cal, n_test, report):
    """Latency predictor (Sec. 5.1) and search (Sec. 5.2) on ViT-L/16 at 384 px,
    batch 32: the LUT of every (linear shape, N:8 pattern) from this library's
    GEMMs (mean of repeated runs), whole-chain measurements of random layer-wise
    configurations, the NNLS calibration of Eq. 1 on some of them and its
    prediction error on the others; then Algorithm 1 on the calibrated
    predictor with a synthetic accuracy stand-in, and the measured latency of
    the configurations it returns."""
    from paper_2607_12505_amd import latency as lt
    from paper_2607_12505_amd import nmsearch
    shapes = lt.vit_large_layer_shapes()
    L = len(shapes)
    pats = list(lt.FAMILY_N8) + [(1, 4), (2, 4)]
    t0 = time.perf_counter()
    cb = lt.ChainBench(torch, shapes, pats, nmspmm.NM_OUT_I32, seed=4)
    log(f"prepared {len(cb.calls)} GEMMs in {time.perf_counter() - t0:.1f} s")
    cb.lut(reps=3, cold=False)                       # warm-up pass
    table, lut_s = cb.lut(reps=20, cold=True)
    hot, _ = cb.lut(reps=20, cold=False)
    log(f"LUT of {len(table)} entries built in {lut_s:.2f} s")
    names = {(8, 8): "dense"}
    pname = lambda p: names.get(p, f"{p[0]}:{p[1]}")
    family = {}
    for which, tab in (("hot", hot), ("cold", table)):
        family[which] = {}
        for shape, lin in zip(shapes[:4], ("qkv", "proj", "fc1", "fc2")):
            m, k, n = shape
            dense_us = tab[(shape, (8, 8))]
            family[which][lin] = {"m": m, "k": k, "n": n, "patterns": {
                pname(p): {"us": round(tab[(shape, p)], 2),
                           "tops": round(2.0 * m * n * k / (tab[(shape, p)] * 1e-6) / 1e12, 1),
                           "speedup_vs_dense": round(dense_us / tab[(shape, p)], 3)} for p in pats}}
    cal = lt.random_assignments(n_cal, L, lt.FAMILY_N8, seed=1)
    test = lt.random_assignments(n_test, L, lt.FAMILY_N8, seed=2)
    test += [[p] * L for p in lt.FAMILY_N8]            # the uniform configurations
    test.append(wl.vit_large_assignment())            # the layer-wise draw of the ViT-L chain workload
    t0 = time.perf_counter()
    T_cal = np.array([cb.measure(a) for a in cal])
    T_test = np.array([cb.measure(a) for a in test])
    log(f"{len(cal) + len(test)} chains measured in {time.perf_counter() - t0:.1f} s")
    # the chain workload's own layer-wise draw (the last test configuration)
    draw = {"measured_us": round(float(T_test[-1]), 1),                # the all-dense chain is T_test[-2]
            "speedup_vs_dense": round(float(T_test[-2] / T_test[-1]), 3)}
    luts = {"cold": table, "hot": hot}
    R_cal = {k: np.array([cb.layer_times(t, a) for a in cal]) for k, t in luts.items()}
    R_test = {k: np.array([cb.layer_times(t, a) for a in test]) for k, t in luts.items()}
    kind = np.arange(L) % 4

    def fit(R, T, structure):
        """Eq. 1 by NNLS: one gamma per layer (as written), or one per linear
        type shared by its 24 layers (4 + 1 unknowns: better posed when few
        configurations are measured)."""
        if structure == "layer":
            return nmsearch.latency_fit(R, T)
        g, b = nmsearch.latency_fit(np.stack([R[:, kind == j].sum(axis=1) for j in range(4)], axis=1), T)
        return g[kind], b

    def errors(gamma, b, R, T):
        pred = np.array([nmsearch.latency_predict(r, gamma, b) for r in R])
        e = np.abs(pred - T) / T
        return {"mean_abs_pct": round(float(e.mean() * 100), 2), "max_abs_pct": round(float(e.max() * 100), 2),
                "within_5pct": round(float((e <= 0.05).mean()), 3)}

    fits = {}
    for lk in ("cold", "hot"):
        fits[f"{lk} LUT, sum without calibration"] = errors(np.ones(L), 0.0, R_test[lk], T_test)
    for lk in ("cold", "hot"):
        for structure in ("layer", "type"):
            for K in sorted({8, 16, 32, len(cal)}):
                if K <= len(cal):
                    g, b = fit(R_cal[lk][:K], T_cal[:K], structure)
                    fits[f"{lk} LUT, gamma per {structure}, {K} configs"] = errors(g, b, R_test[lk], T_test)
    # the predictor the search uses: the variant with the smallest 4-fold
    # cross-validated error on the calibration configurations alone
    folds = np.arange(len(cal)) % 4
    cv = {}
    for lk in ("cold", "hot"):
        for structure in ("layer", "type"):
            errs = []
            for f in range(4):
                g, b = fit(R_cal[lk][folds != f], T_cal[folds != f], structure)
                pred = np.array([nmsearch.latency_predict(r, g, b) for r in R_cal[lk][folds == f]])
                errs += list(np.abs(pred - T_cal[folds == f]) / T_cal[folds == f])
            cv[(lk, structure)] = float(np.mean(errs))
    lut_kind, structure = min(cv, key=cv.get)
    gamma, b = fit(R_cal[lut_kind], T_cal, structure)
    chosen = {"lut": lut_kind, "gamma": structure, "cv_mean_abs_pct": round(cv[(lut_kind, structure)] * 100, 2),
              "test": errors(gamma, b, R_test[lut_kind], T_test)}
    table = luts[lut_kind]
    log(json.dumps(fits))
    log(json.dumps(chosen))

    # Algorithm 1 on the calibrated predictor (largest calibration set)
    lut8 = np.array([[table[(shape, (N, 8))] for N in range(1, 9)] for shape in shapes])
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([5, 5])))
    sens = rng.uniform(0.05, 1.0, L)
    acc_tab = [[float(sens[l] * np.log(N / 8.0)) for N in range(1, 9)] for l in range(L)]

    def accuracy(cfg):
        return sum(acc_tab[l][cfg[l] - 1] for l in range(L))

    lo = nmsearch.latency_predict(lut8[:, 0], gamma, b)
    hi = nmsearch.latency_predict(lut8[:, 7], gamma, b)
    searches = []
    for f in (0.3, 0.6, 0.9):
        target_speedup = 1.0 + (hi / lo - 1.0) * f
        target = hi / target_speedup
        t0 = time.perf_counter()
        cfg, fit, trace = nmsearch.search(lut8, gamma, b, target, accuracy, generations=30, offspring=8,
                                          overshoot=4, seed=7)
        wall = time.perf_counter() - t0
        assign = [(n, 8) for n in cfg]
        pred = nmsearch.latency_predict([lut8[l][cfg[l] - 1] for l in range(L)], gamma, b)
        meas = cb.measure(assign, reps=5)
        counts = {str(N): int(sum(1 for v in cfg if v == N)) for N in range(1, 9)}
        searches.append({"target_speedup": round(target_speedup, 3), "target_us": round(target, 1),
                         "predicted_us": round(pred, 1), "measured_us": round(meas, 1),
                         "measured_speedup_vs_dense": round(T_test[len(test) - 2] / meas, 3),
                         "pred_error_pct": round(abs(pred - meas) / meas * 100, 2),
                         "fitness": round(fit, 4), "fitness_first_last": [round(trace[0], 4), round(trace[-1], 4)],
                         "layers_per_N": counts, "search_s": round(wall, 2)})
        log(json.dumps(searches[-1]))
    res = {"workload": "vit_large_384_b32 linears (96 GEMMs, int32 outputs)", "lut_entries": len(table),
           "lut_build_s": round(lut_s, 2), "calibration_configs": len(cal), "test_configs": len(test),
           "chain_dense_us": round(float(T_test[len(test) - 2]), 1), "fits": fits, "predictor": chosen,
           "family": family, "search": searches, "workload_draw": draw}
    if report:
        write_predictor_report(res, report)
    return res


def write_predictor_report(res, path):
    md = ["# Latency predictor and layer-wise search: ViT-L/16 384 px, batch 32", "",
          "Command: `python3 bench.py --predictor --report profiles/predictor_vit_large.md` (repository root).", "",
          f"LUT: {res['lut_entries']} (shape, pattern) entries, mean of 20 runs each, built in "
          f"{res['lut_build_s']} s (each run starts with flushed caches; the hot LUT of back-to-back repeats is "
          f"shown for comparison).  Calibration on {res['calibration_configs']} random layer-wise N:8 "
          f"configurations, prediction error on {res['test_configs']} others (random, the eight uniform ones and "
          f"the seeded layer-wise draw of the chain workload).  All-dense chain: {res['chain_dense_us']} us; the "
          f"chain workload's seeded layer-wise draw: {res['workload_draw']['measured_us']} us "
          f"({res['workload_draw']['speedup_vs_dense']}x).", "",
          "| fit | mean abs error % | max abs error % | share within 5% |", "|---|---:|---:|---:|"]
    for k, v in res["fits"].items():
        md.append(f"| {k} | {v['mean_abs_pct']} | {v['max_abs_pct']} | {v['within_5pct']} |")
    c = res["predictor"]
    md += ["", f"Predictor used by the search (smallest 4-fold cross-validated error on the calibration "
           f"configurations): {c['lut']} LUT, gamma per {c['gamma']}; cross-validated mean error "
           f"{c['cv_mean_abs_pct']}%, on the test configurations {c['test']['mean_abs_pct']}% mean, "
           f"{c['test']['max_abs_pct']}% max, {c['test']['within_5pct']} within 5%.", "",
           ]
    for which, how in (("hot", "back-to-back repeats, as the linears of a chain run"),
                       ("cold", "caches flushed before every run")):
        fam = res["family"][which]
        pnames = next(iter(fam.values()))["patterns"]
        md += [f"N:8 family per linear from the {which} LUT ({how}; mean us; dense-equivalent TOPS; speedup over "
               f"the dense GEMM):", "",
               "| linear | m | k | n | " + " | ".join(pnames) + " |",
               "|---|---:|---:|---:|" + "---:|" * len(pnames)]
        for lin, f in fam.items():
            md.append(f"| {lin} | {f['m']} | {f['k']} | {f['n']} | " + " | ".join(
                f"{v['us']} / {v['tops']} / {v['speedup_vs_dense']}x" for v in f["patterns"].values()) + " |")
        md.append("")
    md += ["Algorithm 1 on the calibrated predictor (30 generations, 8 offspring, overshoot 4, synthetic "
           "accuracy stand-in), then the returned configuration measured:", "",
           "| target speedup | target us | predicted us | measured us | measured speedup | error % | layers per N (1..8) | search s |",
           "|---:|---:|---:|---:|---:|---:|---|---:|"]
    for s in res["search"]:
        md.append(f"| {s['target_speedup']} | {s['target_us']} | {s['predicted_us']} | {s['measured_us']} | "
                  f"{s['measured_speedup_vs_dense']} | {s['pred_error_pct']} | "
                  f"{' '.join(s['layers_per_N'][str(n)] and str(s['layers_per_N'][str(n)]) or '0' for n in range(1, 9))} | {s['search_s']} |")
    with open(path, "w") as f:
        f.write("\n".join(md) + "\n")


def chaining_experiment(torch, report):
    """INT8 chaining steps (Sec. 6.3 deployment): the requantisation epilogue
    (int8 output) against the int32 and fp16 outputs of the same GEMMs, 2:4
    and dense, on DeiT-S batch 64 and ViT-L batch 32 linears; and the binary16
    activation quantiser on a ViT-L activation tensor.  Mean of 20 runs;
    achieved HBM bandwidth from the algorithmic bytes."""
    from paper_2607_12505_amd import latency as lt
    shapes = [("DeiT-S qkv", 12608, 384, 1152), ("DeiT-S fc1", 12608, 384, 1536), ("DeiT-S fc2", 12608, 1536, 384),
              ("ViT-L fc1", 18464, 1024, 4096), ("ViT-L fc2", 18464, 4096, 1024)]
    rows = []
    for name, m, k, n in shapes:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([31, m, k, n])))
        X = torch.from_numpy(wl.gen_x(m, k, rng)).cuda()
        W, scale = wl.gen_w(n, k, 2, 4, rng)
        dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4))
        Wd = torch.from_numpy(W).cuda()
        sc = torch.from_numpy(scale).cuda()
        qs = torch.full((n,), 1e-3, dtype=torch.float32, device="cuda")
        Y = torch.empty((m, n), dtype=torch.int32, device="cuda")
        Yh = torch.empty((m, n), dtype=torch.int16, device="cuda")
        Yq = torch.empty((m, n), dtype=torch.int8, device="cuda")
        g = wl.Gemm(name, m, k, n, 2, 4)
        for mode, kw, ob in (("int32", dict(Y=Y), 4), ("fp16", dict(Yh=Yh, scale=sc), 2),
                             ("int8", dict(Yq=Yq, qscale=qs), 1)):
            for kind in ("2:4", "dense"):
                if kind == "2:4":
                    fn = lambda kw=kw: nmspmm.spmm(X, dw, **kw)
                    wbytes = algorithmic_bytes(g, False, False) - m * k
                else:
                    fn = lambda kw=kw: nmspmm.gemm_i8_dense(X, Wd, **kw)
                    wbytes = n * k
                us = lt.time_launches(torch, fn, 20)
                b = m * k + wbytes + ob * m * n + (4 * n if mode != "int32" else 0)
                rows.append({"gemm": name, "m": m, "k": k, "n": n, "output": mode, "kind": kind,
                             "us": round(us, 2), "gbs": round(b / us / 1e3, 1),
                             "hbm_frac": round(b / us / 1e3 / PEAK_HBM_GBS, 3)})
                log(json.dumps(rows[-1]))
    count = 18464 * 1024
    x = torch.randn(count, dtype=torch.float16, device="cuda").view(torch.int16)
    xq = torch.empty(count, dtype=torch.int8, device="cuda")
    us = lt.time_launches(torch, lambda: nmspmm.quantize_f16(x, 1.0 / 0.05, xq=xq), 20)
    quant = {"elements": count, "us": round(us, 2), "gbs": round(3 * count / us / 1e3, 1),
             "hbm_frac": round(3 * count / us / 1e3 / PEAK_HBM_GBS, 3)}
    log(json.dumps(quant))
    res = {"requant_epilogue": rows, "quantize_f16": quant}
    if report:
        md = ["# INT8 chaining: requantisation epilogue and activation quantiser", "",
              "Command: `python3 bench.py --chaining --report profiles/int8_chaining.md` (repository root).  "
              "Mean of 20 back-to-back runs per row (HIP events); GB/s from the algorithmic bytes (X, the weight "
              "-- compact packed form for 2:4 --, the output, the multipliers).", "",
              "| GEMM | m | k | n | output | weight | us | GB/s | HBM fraction |", "|---|---:|---:|---:|---|---|---:|---:|---:|"]
        for r in rows:
            md.append(f"| {r['gemm']} | {r['m']} | {r['k']} | {r['n']} | {r['output']} | {r['kind']} | {r['us']} | "
                      f"{r['gbs']} | {r['hbm_frac']} |")
        md += ["", f"Activation quantiser (binary16 -> int8, {count} elements = one ViT-L fc1 input): "
               f"{quant['us']} us, {quant['gbs']} GB/s ({quant['hbm_frac']} of HBM peak)."]
        with open(report, "w") as f:
            f.write("\n".join(md) + "\n")
    return res


def paper_grid(torch, report):
    """The paper's kernel benchmark grid (Sec. 6.1): tokens m in {64, 128, 256,
    512}, n and k in {128, 256, 512, 1024}, sparsity 50 / 75 / 87.5 % (2:4 and
    4:8 / 1:4 and 2:8 / 1:8).  Each case: this library's sparse GEMM, its dense
    MFMA GEMM, and the vendor dense INT8 GEMM (hipBLASLt through
    torch._int_mm, a measured reference only), int32 output, mean of 50
    back-to-back runs."""
    from paper_2607_12505_amd import latency as lt
    sizes = (128, 256, 512, 1024)
    rows = []
    for m in (64, 128, 256, 512):
        for n in sizes:
            for k in sizes:
                rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([6, m, n, k])))
                X = torch.from_numpy(wl.gen_x(m, k, rng)).cuda()
                Y = torch.empty((m, n), dtype=torch.int32, device="cuda")
                Wd_host, _ = wl.gen_w(n, k, 8, 8, rng)
                Wd = torch.from_numpy(Wd_host).cuda()
                WdT = Wd.t().contiguous()
                t_dense = lt.time_launches(torch, lambda: nmspmm.gemm_i8_dense(X, Wd, Y=Y), 50)
                t_vendor = lt.time_launches(torch, lambda: torch._int_mm(X, WdT), 50)
                for (N, M), spars in (((2, 4), 50), ((4, 8), 50), ((1, 4), 75), ((2, 8), 75), ((1, 8), 87.5)):
                    W, _ = wl.gen_w(n, k, N, M, rng)
                    dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, N, M))
                    t_sp = lt.time_launches(torch, lambda: nmspmm.spmm(X, dw, Y=Y), 50)
                    rows.append({"m": m, "n": n, "k": k, "pattern": f"{N}:{M}", "sparsity": spars,
                                 "sparse_us": round(t_sp, 2), "dense_us": round(t_dense, 2),
                                 "vendor_us": round(t_vendor, 2)})
        log(f"grid m={m} done")
    summary = {}
    for key in ("50", "75", "87.5", "all"):
        sel = [r for r in rows if key == "all" or float(r["sparsity"]) == float(key)]
        summary[key] = {
            "cases": len(sel),
            "mean_speedup_vs_own_dense": round(float(np.mean([r["dense_us"] / r["sparse_us"] for r in sel])), 3),
            "mean_speedup_vs_vendor_dense": round(float(np.mean([r["vendor_us"] / r["sparse_us"] for r in sel])), 3),
        }
    log(json.dumps(summary))
    if report:
        md = ["# The paper's kernel benchmark grid on MI355X", "",
              "Command: `python3 bench.py --paper-grid --report profiles/paper_grid.md` (repository root).  Tokens m in "
              "{64, 128, 256, 512}, n and k in {128, 256, 512, 1024}; 50 % = 2:4 and 4:8, 75 % = 1:4 and 2:8, 87.5 % "
              "= 1:8; int32 output; mean of 50 back-to-back runs with inputs resident (HIP events).  \"vendor\" = the "
              "dense INT8 GEMM of hipBLASLt through torch._int_mm, timed as a reference.", "",
              "| sparsity | cases | mean speedup vs this library's dense MFMA GEMM | mean speedup vs the vendor dense GEMM |",
              "|---|---:|---:|---:|"]
        for key, v in summary.items():
            md.append(f"| {key} | {v['cases']} | {v['mean_speedup_vs_own_dense']} | {v['mean_speedup_vs_vendor_dense']} |")
        md += ["", "| m | n | k | pattern | sparse us | dense us | vendor dense us |", "|---:|---:|---:|---|---:|---:|---:|"]
        for r in rows:
            md.append(f"| {r['m']} | {r['n']} | {r['k']} | {r['pattern']} | {r['sparse_us']} | {r['dense_us']} | "
                      f"{r['vendor_us']} |")
        with open(report, "w") as f:
            f.write("\n".join(md) + "\n")
    return {"summary": summary, "rows": len(rows)}


def shape_report(torch, report, cfgs=(0, 1, 2, 3, 4)):
    """Per-shape roofline of every workload GEMM (distinct shape and pattern):
    sparse and dense time, the compute and HBM fractions against the data-sheet
    peaks, the compute fraction against the matrix-instruction rate measured in
    the same run on random operands, and the roofline fraction (the binding
    one).  Times: mean of 5 back-to-back launches, inputs resident."""
    from paper_2607_12505_amd import latency as lt
    ceil = mfma_ceiling(torch)
    sp_rate = ceil["smfmac_i32_16x16x128_i8_random_pops"] * 1e3       # dense-equivalent TOPS
    dn_rate = ceil["mfma_i32_16x16x64_i8_random_pops"] * 1e3
    rows = []
    for cfg in cfgs:
        work = wl.workload(cfg)
        seen, gemms = set(), []
        for g in work.gemms:
            key = (g.m, g.k, g.n, g.N, g.M)
            if key not in seen:
                seen.add(key)
                gemms.append(g)
        xd, xh = {}, {}
        preps = [Prepared(cfg, g, xd, xh, work.out_int32, work.out_f16, torch, use_dense_kernel=(g.N == g.M))
                 for g in gemms]
        torch.cuda.synchronize()
        each = time_each(preps, torch)
        outs = ("int32" if work.out_int32 else "") + ("+fp16" if work.out_f16 else "")
        # the vendor dense INT8 GEMM (hipBLASLt through torch._int_mm, int32
        # output) beside ours, where the outputs are the same (int32 only)
        vendor = []
        for p in preps:
            if work.out_f16 or not work.out_int32:
                vendor.append(None)
                continue
            WdT = p.Wd.t().contiguous()
            try:
                vendor.append(lt.time_launches(torch, lambda: torch._int_mm(p.Xd, WdT), 5) * 1e-3)
            except RuntimeError:
                vendor.append(None)
            del WdT
        for p, (ts, td), tv in zip(preps, each, vendor):
            g, kind = p.g, p.splan.kind
            ops = g.dense_eq_ops
            peak = PEAK_SPARSE_TOPS if kind == nmspmm.NM_KIND_SP42 else PEAK_INT8_TOPS
            rate = sp_rate if kind == nmspmm.NM_KIND_SP42 else sp_rate / 2 if kind == nmspmm.NM_KIND_SP42X2 \
                else dn_rate
            b = algorithmic_bytes(g, work.out_int32, work.out_f16, sparse=p.sparse_kernel)
            bd = algorithmic_bytes(g, work.out_int32, work.out_f16, sparse=False)
            t_mfma, t_hbm = ops / (peak * 1e9), b / (PEAK_HBM_GBS * 1e6)      # ms
            td_mfma, td_hbm = ops / (PEAK_INT8_TOPS * 1e9), bd / (PEAK_HBM_GBS * 1e6)
            rows.append({"workload": work.name, "gemm": g.name, "m": g.m, "k": g.k, "n": g.n, "pattern": pattern_name(g),
                         "outputs": outs, "kernel": p.kernel_name(p.splan), "sparse_us": ts * 1e3, "dense_us": td * 1e3,
                         "speedup": td / ts, "tops": ops / (ts * 1e-3) / 1e12,
                         "bound": "mfma" if t_mfma > t_hbm else "hbm",
                         "mfma_frac": t_mfma / ts, "mfma_frac_measured": ops / (rate * 1e9) / ts,
                         "hbm_gbs": b / (ts * 1e-3) / 1e9, "hbm_frac": t_hbm / ts, "roofline_frac": max(t_mfma, t_hbm) / ts,
                         "dense_roofline_frac": max(td_mfma, td_hbm) / td,
                         "vendor_us": tv * 1e3 if tv is not None else None})
        log(f"shape report: {work.name} done ({len(preps)} shapes)")
        del preps
        torch.cuda.empty_cache()
    if report:
        md = ["# Per-shape roofline of the workload GEMMs", "",
              "Command: `python3 bench.py --shape-report --report profiles/per_shape_roofline.md` (repository root).  "
              "Every distinct (shape, N:M) of the five workloads; mean of 5 back-to-back launches with inputs resident "
              "(HIP events).  Peaks: HBM 8 TB/s; matrix cores 10.07 dense-equivalent POPS for one 4:2 stream "
              "(smfmac), 5.03 POPS for two streams and dense.  \"MFMA frac (meas.)\" divides by the rate measured "
              f"in the same run on random int8 operands: smfmac {ceil['smfmac_i32_16x16x128_i8_random_pops']} "
              f"dense-equivalent POPS (two streams: half), dense {ceil['mfma_i32_16x16x64_i8_random_pops']} POPS "
              f"(on zeros: {ceil['smfmac_i32_16x16x128_i8_zero_pops']} and {ceil['mfma_i32_16x16x64_i8_zero_pops']}).  "
              "Roofline fraction = max(compute time at peak, algorithmic bytes at 8 TB/s) / measured time; "
              "algorithmic bytes count the compact packed weight (N/M of the values plus ceil(log2 M) bits per value).  "
              "Each row has its own input and output buffers; the dense time of one shape, measured again in every "
              "pattern row, shows the run-to-run spread (largest on the biggest outputs).  \"vendor dense\": the dense "
              "INT8 GEMM of hipBLASLt through torch._int_mm (int32 output, so only for the int32-only workloads), "
              "timed beside ours as a reference for the dense baseline.", "",
              "| workload | GEMM | m | k | n | N:M | out | sparse kernel | sparse us | dense us | speedup | TOPS | bound | "
              "MFMA frac | MFMA frac (meas.) | GB/s | HBM frac | roofline frac | dense roofline frac | vendor dense us |",
              "|---|---|---:|---:|---:|---|---|---|---:|---:|---:|---:|---|---:|---:|---:|---:|---:|---:|---:|"]
        for r in rows:
            md.append(f"| {r['workload']} | {r['gemm']} | {r['m']} | {r['k']} | {r['n']} | {r['pattern']} | {r['outputs']} "
                      f"| `{r['kernel']}` | {r['sparse_us']:.1f} | {r['dense_us']:.1f} | {r['speedup']:.2f} | "
                      f"{r['tops']:.0f} | {r['bound']} | {r['mfma_frac']:.3f} | {r['mfma_frac_measured']:.3f} | "
                      f"{r['hbm_gbs']:.0f} | {r['hbm_frac']:.3f} | {r['roofline_frac']:.3f} | "
                      f"{r['dense_roofline_frac']:.3f} | "
                      f"{'—' if r['vendor_us'] is None else format(r['vendor_us'], '.1f')} |")
        with open(report, "w") as f:
            f.write("\n".join(md) + "\n")
    fr = np.array([r["roofline_frac"] for r in rows])
    vd = [(r["vendor_us"], r["dense_us"]) for r in rows if r["vendor_us"] is not None]
    return {"shapes": len(rows), "roofline_frac_median": round(float(np.median(fr)), 3),
            "dense_vs_vendor_median": round(float(np.median([v / d for v, d in vd])), 3) if vd else None,
            "roofline_frac_min": round(float(fr.min()), 3), "roofline_frac_max": round(float(fr.max()), 3),
            "mfma_measured": ceil}


def graph_layer(torch, reps: int = 200) -> dict:
    """One DeiT-Base layer's four linears (qkv, proj, fc1, fc2; 2:4, int32
    output) at batch 1 and 8, launched from Python one call at a time as an
    application would (no pre-queued sleep), against the same four calls
    captured once in a HIP graph and replayed: mean microseconds per layer."""
    res = {}
    E = torch.cuda.Event
    for batch in (1, 8):
        m = 197 * batch
        rng = np.random.default_rng(batch)
        calls = []
        for k, n in ((768, 2304), (768, 768), (768, 3072), (3072, 768)):
            X = torch.from_numpy(wl.gen_x(m, k, rng)).cuda()
            W, _ = wl.gen_w(n, k, 2, 4, rng)
            dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4))
            Y = torch.empty((m, n), dtype=torch.int32, device="cuda")
            calls.append(lambda X=X, dw=dw, Y=Y: nmspmm.spmm(X, dw, Y=Y))

        def layer():
            for c in calls:
                c()
        for _ in range(3):
            layer()
        torch.cuda.synchronize()
        e0, e1 = E(enable_timing=True), E(enable_timing=True)
        e0.record()
        for _ in range(reps):
            layer()
        e1.record()
        torch.cuda.synchronize()
        eager_us = e0.elapsed_time(e1) * 1e3 / reps
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            layer()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            layer()
        g.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        graph_us = e0.elapsed_time(e1) * 1e3 / reps
        res[f"b{batch}"] = {"m": m, "eager_us_per_layer": round(eager_us, 2), "graph_us_per_layer": round(graph_us, 2)}
    return res


def write_sweep_report(sweep_json, path):
    """Markdown table of a planner evaluation written by --sweep-out."""
    d = json.load(open(sweep_json))
    s = d["summary"]
    md = ["# Planner evaluation (Table-1 methodology) on MI355X", "",
          "Commands: `python3 bench.py --sweep 0,1,2,3,4 --sweep-out sweep.json` (GPU; every (tile, split_k) "
          "candidate timed in two passes of 10 launches each (the second pass in reverse order, each behind a 1 ms "
          "spin), the faster pass kept, outputs rotated over at least two "
          "buffers and at least 512 MB in all, twice the last-level cache), "
          "then `python3 bench.py --sweep-report sweep.json --report <this file>`.", "",
          "Normalised performance = t(sweep optimum) / t(planner choice); tile indices are those of the "
          "library's tile table (`nm_tile_info`).", "",
          f"Summary, sparse GEMMs: {s['cases']} distinct (shape, N:M) cases; planner Top-1 hit rate "
          f"{s['top1_hit_rate']}, average normalised performance {s['avg_norm_perf']}, worst {s['worst_norm_perf']}; "
          f"gain over a fixed split_k = 1 with the same tile {s['gain_over_fixed_split1']}.", ""]
    gs = d.get("grid_summary")
    if gs:
        md += ["The paper's kernel grid (Sec. 6.1: m in {64, 128, 256, 512}, n and k in {128, 256, 512, 1024}; int32 "
               "output), per sparsity as in Table 1:", "",
               "| sparsity | cases | Top-1 hit rate | average normalised | worst normalised | gain over a fixed "
               "128x128 plan |", "|---|---:|---:|---:|---:|---:|"]
        for key, v in gs.items():
            if v:
                label = "dense baseline" if key == "dense" else f"{key} %"
                md.append(f"| {label} | {v['cases']} | {v['top1_hit_rate']} | {v['avg_norm_perf']} | "
                          f"{v['worst_norm_perf']} | {v.get('gain_over_fixed_128x128')} |")
        md.append("")
    ds = d.get("dense_summary")
    if ds:
        md += [f"Dense INT8 baseline (every sparse shape's dense counterpart and the dense layers of the chain): "
               f"{ds['cases']} distinct shapes; planner Top-1 hit rate {ds['top1_hit_rate']}, average normalised "
               f"performance {ds['avg_norm_perf']}, worst {ds['worst_norm_perf']}.", ""]
    md += ["| workload | m | k | n | N:M | planner tile/split | us | best tile/split | us | norm |",
           "|---|---:|---:|---:|---|---|---:|---|---:|---:|"]
    for r in d["rows"]:
        md.append(f"| cfg{r['cfg']} {r['gemm']} | {r['m']} | {r['k']} | {r['n']} | {r['pattern']} | "
                  f"{r['planned'][0]}/{r['planned'][1]} | {r['t_planned_us']:.1f} | {r['best'][0]}/{r['best'][1]} | "
                  f"{r['t_best_us']:.1f} | {r['t_best_us'] / r['t_planned_us']:.3f} |")
    with open(path, "w") as f:
        f.write("\n".join(md) + "\n")


KERNEL_SOURCE = os.path.join(ROOT, "paper_2607_12505_amd", "csrc", "nmspmm_kernels.hip")


def kernel_source_sha256():
    """SHA-256 of the kernel source with comments and blank space removed, so
    that a counter record stays valid across edits that change no code."""
    import hashlib
    import re
    src = open(KERNEL_SOURCE).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = re.sub(r"\s+", " ", src).strip()
    return hashlib.sha256(src.encode()).hexdigest()


def default_traffic_path(workload_name):
    return os.path.join(ROOT, "profiles", f"traffic_{workload_name}.json")


def rocprof_summary(trace_dir, fetch_dir, write_dir, bench_json, copy_mib, commands, out_md, sq_dir=None):
    """Summarises rocprofv3 CSV output of a bench run: per-kernel durations
    from the kernel trace, and FETCH_SIZE / WRITE_SIZE per dispatch scaled by
    what the same counters read for the calibration copy (copy_mib MiB read
    and written); with sq_dir, also matrix-core busy time and LDS bank
    conflicts per kernel (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE,
    SQ_LDS_BANK_CONFLICT, SQ_LDS_IDX_ACTIVE).  Writes a markdown summary and the
    traffic record of the dominant kernel next to it."""
    import csv
    import glob
    line = json.loads(open(bench_json).read().strip().splitlines()[-1])
    dom = line["roofline"]["kernel"]
    work = line["config"]["workload"]
    stats = list(csv.DictReader(open(glob.glob(os.path.join(trace_dir, "*_kernel_stats.csv"))[0])))
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))

    def counters(d, name=None):
        per = {}
        for r in csv.DictReader(open(glob.glob(os.path.join(d, "*_counter_collection.csv"))[0])):
            if name is None or r["Counter_Name"] == name:
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return per

    fetch, write = counters(fetch_dir), counters(write_dir)
    calib = [k for k in fetch if "neg_kernel" in k]
    if len(calib) != 1:
        raise SystemExit("calibration copy kernel not found in the counter output")
    true_bytes = copy_mib * (1 << 20)
    f_scale = true_bytes / (np.mean(fetch[calib[0]]) * 1024)
    w_scale = true_bytes / (np.mean(write[calib[0]]) * 1024)

    def find(per, name):
        ks = [k for k in per if name in k]
        return per[ks[0]] if ks else None

    dom_fetch, dom_write = find(fetch, dom), find(write, dom)
    bytes_per_launch = (np.mean(dom_fetch) * 1024 * f_scale + np.mean(dom_write) * 1024 * w_scale)
    dom_stats = [r for r in stats if dom in r["Name"]][0]
    md = [f"# rocprofv3 summary: `{dom}` on workload `{work}`", ""]
    md += ["Commands (repository root as working directory of the bench; rocprofv3 run from /tmp):", "", "```"]
    md += commands + ["```", ""]
    md += [f"Dominant sparse kernel: `{dom}`: {dom_stats['Calls']} calls, average "
           f"{float(dom_stats['AverageNs']) / 1e3:.2f} us (min {float(dom_stats['MinNs']) / 1e3:.2f}, "
           f"max {float(dom_stats['MaxNs']) / 1e3:.2f}); bench.py HIP-event average over the timed region: "
           f"{line['roofline']['avg_launch_us']:.2f} us.", ""]
    md += ["| kernel | calls | avg us | total ms |", "|---|---:|---:|---:|"]
    for r in stats[:14]:
        md.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['TotalDurationNs']) / 1e6:.3f} |")
    md += ["", "HBM traffic per dispatch (FETCH_SIZE and WRITE_SIZE, KiB, scaled by the calibration copy of "
           f"{copy_mib} MiB read + {copy_mib} MiB written: fetch x{f_scale:.3f}, write x{w_scale:.3f}):", "",
           "| kernel | dispatches | FETCH KiB | WRITE KiB | scaled MB |", "|---|---:|---:|---:|---:|"]
    for k in sorted(set(fetch) & set(write), key=lambda k: -np.mean(write[k]))[:10]:
        mb = (np.mean(fetch[k]) * 1024 * f_scale + np.mean(write[k]) * 1024 * w_scale) / 1e6
        md.append(f"| `{k[:90]}` | {len(fetch[k])} | {np.mean(fetch[k]):.0f} | {np.mean(write[k]):.0f} | {mb:.2f} |")
    alg = line["roofline"]["algorithmic_bytes_per_launch"]
    md += ["", f"Dominant kernel: measured traffic {bytes_per_launch / 1e6:.2f} MB per launch vs "
           f"{alg / 1e6:.2f} MB algorithmic ({bytes_per_launch / alg:.3f}x)."]
    if sq_dir:
        busy, active = counters(sq_dir, "SQ_VALU_MFMA_BUSY_CYCLES"), counters(sq_dir, "GRBM_GUI_ACTIVE")
        conf, lds = counters(sq_dir, "SQ_LDS_BANK_CONFLICT"), counters(sq_dir, "SQ_LDS_IDX_ACTIVE")
        simds, xcds = 1024, 8   # MI355X: 256 CUs x 4 SIMDs, in 8 XCDs
        md += ["", "Matrix cores and LDS per dispatch (one more pass: `--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
               "SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE`).  GRBM_GUI_ACTIVE is reported summed over the 8 XCDs, so "
               f"MFMA busy = busy cycles / (GRBM_GUI_ACTIVE / {xcds} x {simds} SIMDs), the definition of rocprofv3's "
               "MfmaUtil; LDS bank conflicts = conflict cycles / LDS active cycles:", "",
               "| kernel | dispatches | MFMA busy % | LDS conflict % |", "|---|---:|---:|---:|"]
        for k in sorted(busy, key=lambda k: -np.mean(busy[k])):
            if "nmspmm" not in k or k not in active:
                continue
            mb = 100.0 * np.mean(busy[k]) / (np.mean(active[k]) / xcds * simds)
            lc = 100.0 * np.mean(conf[k]) / max(np.mean(lds[k]), 1.0) if k in conf and k in lds else float("nan")
            md.append(f"| `{k[:90]}` | {len(busy[k])} | {mb:.1f} | {lc:.2f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(md) + "\n")
    rec = {"kernel": dom, "workload": work, "bytes_per_launch": int(bytes_per_launch),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "kernel_source_sha256": kernel_source_sha256(), "summary": os.path.basename(out_md)}
    with open(default_traffic_path(work), "w") as f:
        json.dump(rec, f, indent=1)
    print("\n".join(md))


def cache_state(preps) -> str:
    """What the caches hold when a GEMM of the timed steps starts: every step
    reuses the same buffers, but the distinct bytes one step touches (inputs,
    weights and outputs of every sparse and dense GEMM) decide whether the
    previous step left them in the 256 MB MALL and the 8 x 4 MB of L2."""
    seen, total = set(), 0
    for p in preps:
        tensors = [p.Xd, p.Wd, p.Y, p.Yh, p.Yd, p.Yhd, p.scale]
        if p.sparse_kernel:
            tensors += [p.dw.vals, p.dw.meta]
        for t in tensors:
            if t is not None and t.data_ptr() not in seen:
                seen.add(t.data_ptr())
                total += t.numel() * t.element_size()
    caches = 256e6 + 32e6
    if total > caches:
        return (f"same buffers every step; one step touches {total / 1e9:.2f} GB, over the 288 MB of MALL and L2, "
                "so the caches cannot keep a step's inputs until the next step")
    return f"same buffers every step; one step touches {total / 1e6:.0f} MB, so inputs can stay cache-resident"


def mfma_ceiling(torch, iters: int = 4000, reps: int = 3) -> dict:
    """Matrix-instruction rate this GPU sustains (nm_probe_mfma_rate), in
    dense-equivalent POPS, on uniform random int8 operands and on zeros: the
    practical compute ceiling beside the data-sheet peak (random operands make
    the chip lower its clock)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    g = torch.Generator().manual_seed(2607)
    rnd = torch.randint(-2 ** 31, 2 ** 31, (nmprobe.NM_PROBE_WORDS,), generator=g, dtype=torch.int64)
    rnd = rnd.to(torch.int32).cuda()
    zero = torch.zeros_like(rnd)
    wgs = 4 * cus
    out = torch.empty(wgs * 256, dtype=torch.int32, device="cuda")
    ticks = torch.zeros(2 * wgs, dtype=torch.int64, device="cuda")
    wall_hz = nmprobe.wall_clock_khz() * 1e3
    res = {}
    for kind, name, macs in ((nmspmm.NM_KIND_SP42, "smfmac_i32_16x16x128_i8", 16 * 16 * 128),
                             (nmspmm.NM_KIND_DENSE, "mfma_i32_16x16x64_i8", 16 * 16 * 64)):
        for tname, tab in (("random", rnd), ("zero", zero)):
            nmprobe.probe_mfma_rate(kind, tab, 16, out)
            best, mhz = float("inf"), 0.0
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                nmprobe.probe_mfma_rate(kind, tab, iters, out, ticks)
                e1.record()
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1)
                if ms < best:
                    t = ticks.cpu().numpy().reshape(-1, 2).astype(np.float64)
                    best, mhz = ms, t[:, 0].sum() / (t[:, 1].sum() / wall_hz) / 1e6
            ops = wgs * 4 * iters * 8 * 2 * macs
            res[f"{name}_{tname}_pops"] = round(ops / (best * 1e-3) / 1e15, 3)
            res[f"{name}_{tname}_clock_mhz"] = round(float(mhz))
    res["setup"] = (f"{wgs} workgroups x 4 waves, 8 independent instructions per wave per iteration, {iters} "
                    "iterations; operands uniform random int8 bytes or all zeros; clock = shader cycles over "
                    "real-time counter ticks during the loop")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=1, help="0..4 (default 1: DeiT-Small linears, batch 64)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the DeiT-Base per-batch speedups reported beside the main line")
    ap.add_argument("--no-mfma-ceiling", action="store_true",
                    help="skip the measured matrix-instruction rate reported beside the main line")
    ap.add_argument("--no-store-only", action="store_true",
                    help="skip the output-stream-only launches of the dominant kernel (keeps profiler traces to the "
                         "real launches)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay of the step reported beside the main line")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after timing, run one plain device copy of MIB MiB (profiler counter calibration)")
    ap.add_argument("--sweep", type=str, default=None,
                    help="planner evaluation over the given comma-separated configs (e.g. 0,1,2,3,4); 'grid' adds "
                         "the paper's kernel grid")
    ap.add_argument("--sweep-out", type=str, default=None, help="JSON file for the sweep results")
    ap.add_argument("--sweep-report", type=str, default=None, metavar="SWEEP_JSON",
                    help="markdown report (--report) of a sweep JSON (no GPU needed)")
    ap.add_argument("--traffic", type=str, default=None,
                    help="JSON record of measured HBM bytes per launch of the dominant kernel "
                         "(default: profiles/traffic_<workload>.json, used only if it matches this kernel source)")
    ap.add_argument("--rocprof-summary", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"), default=None,
                    help="summarise rocprofv3 CSV output of a bench run (no GPU needed)")
    ap.add_argument("--bench-json", type=str, default=None, help="bench output line used by --rocprof-summary")
    ap.add_argument("--rocprof-sq", type=str, default=None,
                    help="rocprofv3 counter output with MFMA busy / LDS bank conflict counters (--rocprof-summary)")
    ap.add_argument("--summary-out", type=str, default=None, help="markdown file written by --rocprof-summary")
    ap.add_argument("--commands", type=str, default=None, help="file with the profiling commands to quote")
    ap.add_argument("--predictor", action="store_true",
                    help="latency LUT + Eq. 1 calibration + Algorithm 1 on ViT-L (prints one JSON line)")
    ap.add_argument("--paper-grid", action="store_true",
                    help="the paper's kernel benchmark grid vs the dense GEMMs (prints one JSON line)")
    ap.add_argument("--chaining", action="store_true",
                    help="int8 requantisation epilogue and activation quantiser timings (prints one JSON line)")
    ap.add_argument("--graph-layer", action="store_true",
                    help="DeiT-Base layer at batch 1 and 8: Python launches vs one HIP graph replay (one JSON line)")
    ap.add_argument("--shape-report", action="store_true",
                    help="per-shape roofline of every workload GEMM (prints one JSON line; --report for markdown)")
    ap.add_argument("--cal", type=int, default=64, help="calibration configurations for --predictor")
    ap.add_argument("--test", type=int, default=32, help="random test configurations for --predictor")
    ap.add_argument("--report", type=str, default=None, help="markdown report of --predictor / --chaining")
    args = ap.parse_args()

    if args.sweep_report:
        write_sweep_report(args.sweep_report, args.report)
        return
    if args.rocprof_summary:
        cmds = open(args.commands).read().strip().splitlines() if args.commands else []
        rocprof_summary(*args.rocprof_summary, args.bench_json, args.copy_calibration or 256, cmds,
                        args.summary_out, args.rocprof_sq)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the method is a "
              "single-GPU kernel; how it would shard is a design note, not a measured path)", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    nmspmm.lib()
    torch.cuda.set_device(0)
    if args.sweep:
        summary = sweep([c if c == "grid" else int(c) for c in args.sweep.split(",")], torch, 10, args.sweep_out)
        print(json.dumps({"planner_evaluation": summary}), flush=True)
        return
    if args.chaining:
        print(json.dumps({"chaining": chaining_experiment(torch, args.report)}), flush=True)
        return
    if args.paper_grid:
        print(json.dumps({"paper_grid": paper_grid(torch, args.report)}), flush=True)
        return
    if args.predictor:
        print(json.dumps({"predictor": predictor_experiment(torch, args.cal, args.test, args.report)}), flush=True)
        return
    if args.shape_report:
        print(json.dumps({"shape_report": shape_report(torch, args.report)}), flush=True)
        return
    if args.graph_layer:
        print(json.dumps({"graph_layer": graph_layer(torch)}), flush=True)
        return

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
    groups = launch_groups(preps)
    time_steps(preps, groups, max(1, args.warmup), torch, sleep_cycles)

    torch.cuda.synchronize()
    w0 = time.perf_counter()
    t = time_steps(preps, groups, args.steps, torch, sleep_cycles)
    wall = time.perf_counter() - w0
    ms_per_step = wall * 1e3 / args.steps
    tg = t.mean(axis=0)  # per group: mean over steps (the paper averages repeated runs, Sec. 5.1)
    graph_sparse_ms, graph_dense_ms = (graph_steps(preps, groups, args.steps, torch, sleep_cycles)
                                       if not args.no_graph else (None, None))
    chain = chain_times(preps, torch, max(3, min(args.steps, 10)), sleep_cycles) if work.chain else None

    ops = np.array([p.g.dense_eq_ops for p in preps], np.float64)
    sparse_ms = sum(tg[gi] for gi, ((side, _), _) in enumerate(groups) if side == "sparse")
    dense_ms = sum(tg[gi] for gi, ((side, _), _) in enumerate(groups) if side == "dense")
    value = ops.sum() / (sparse_ms * 1e-3) / 1e12
    dense_tops = ops.sum() / (dense_ms * 1e-3) / 1e12
    speedup = dense_ms / sparse_ms

    # per pattern (detail pass in whole steps ordered by pattern, outside the timed region)
    per_pattern = {}
    for pat, (ts, td) in time_keyed_in_steps(preps, lambda p: pattern_name(p.g), torch, 5).items():
        sel = np.array([pattern_name(p.g) == pat for p in preps])
        per_pattern[pat] = {
            "tops": round(float(ops[sel].sum() / (ts * 1e-3) / 1e12), 1),
            "speedup_vs_dense": round(float(td / ts), 3),
        }

    # dominant kernel: the sparse-side kernel instantiation with the most time per step
    gsum = {}
    for gi, ((side, name), idx) in enumerate(groups):
        if side != "sparse":
            continue
        gsum[name] = {"time_ms": tg[gi], "launches": len(idx),
                      "bytes": sum(algorithmic_bytes(preps[i].g, out_i32, out_f16, sparse=preps[i].sparse_kernel)
                                   for i in idx)}
    dom_name = max(gsum, key=lambda k: gsum[k]["time_ms"])
    dom = gsum[dom_name]
    avg_ms = dom["time_ms"] / dom["launches"]
    dom_idx = next(idx for (side, name), idx in groups if side == "sparse" and name == dom_name)
    store_ms = None if args.no_store_only else store_only_time(preps, dom_idx, torch)
    achieved = dom["bytes"] / dom["launches"] / (avg_ms * 1e-3) / 1e9
    # which roofline binds this kernel: its algorithmic bytes at the HBM peak
    # against its dense-equivalent ops at the matrix-core peak of its kind
    dom_ops = sum(preps[i].g.dense_eq_ops for i in dom_idx)
    peak_ops = PEAK_SPARSE_TOPS if preps[dom_idx[0]].splan.kind == nmspmm.NM_KIND_SP42 else PEAK_INT8_TOPS
    mfma_bound = dom_ops / (peak_ops * 1e12) > dom["bytes"] / (PEAK_HBM_GBS * 1e9)
    traffic = None
    tpath = args.traffic or default_traffic_path(work.name)
    if os.path.exists(tpath):
        with open(tpath) as f:
            tr = json.load(f)
        # counters taken on another kernel (or an older build of it) do not count
        if (tr.get("kernel") == dom_name and tr.get("workload") == work.name
                and tr.get("kernel_source_sha256") == kernel_source_sha256()):
            traffic = tr.get("bytes_per_launch")
    if mfma_bound:
        achieved_ops = dom_ops / dom["launches"] / (avg_ms * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved_ops, 1), "peak": peak_ops, "unit": "TOPS",
                    "frac": round(achieved_ops / peak_ops, 4)}
    else:
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roofline.update({
        "traffic": traffic,
        "kernel": dom_name,
        "launches_per_step": dom["launches"],
        "avg_launch_us": round(avg_ms * 1e3, 2),
        "algorithmic_bytes_per_launch": int(dom["bytes"] / dom["launches"]),
        "algorithmic_ops_per_launch": int(dom_ops / dom["launches"]),
        "hbm_gbs": round(achieved, 1),
    })
    if store_ms is not None:
        # the same launches with the reduction skipped: the ceiling this
        # kernel's own output stream sets (context beside the HBM peak)
        roofline["output_stream_only_us"] = round(store_ms * 1e3, 2)
        roofline["frac_of_output_stream_only"] = round(store_ms / avg_ms, 3)

    # per GEMM, inside whole steps with an event after every GEMM (stderr table only)
    per_gemm = time_keyed_in_steps(preps, lambda p: preps.index(p), torch, 3)
    ts = np.array([per_gemm[i][0] for i in range(len(preps))])
    td = np.array([per_gemm[i][1] for i in range(len(preps))])
    log(f"\n{'gemm':<22}{'m':>7}{'k':>6}{'n':>6}  {'sparse kernel':<30}{'sparse us':>10}{'dense us':>10}"
        f"{'TOPS':>8}{'dTOPS':>8}{'spd':>7}{'GB/s':>8}")
    for i, p in enumerate(preps):
        g = p.g
        b = algorithmic_bytes(g, out_i32, out_f16, sparse=p.sparse_kernel)
        log(f"{g.name:<22}{g.m:>7}{g.k:>6}{g.n:>6}  {p.kernel_name(p.splan) + '/s' + str(p.splan.split_k):<30}"
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
        "sparse_ms_per_step": round(float(sparse_ms), 4),
        # per-step totals: the mean above (the paper averages repeated runs); the median is robust to outliers
        "sparse_ms_per_step_median": round(float(np.median(t[:, [gi for gi, ((sd, _), _) in enumerate(groups)
                                                                  if sd == "sparse"]].sum(axis=1))), 4),
        "cache_state": cache_state(preps),
        "dense_ms_per_step": round(float(dense_ms), 4),
        "roofline": roofline,
    }
    if chain is not None:
        # the layers in network order, one event pair around the whole chain
        line["chain"] = {"sparse_ms": round(chain[0], 4), "dense_ms": round(chain[1], 4),
                         "speedup_vs_dense": round(chain[1] / chain[0], 3),
                         "tops": round(float(ops.sum() / (chain[0] * 1e-3) / 1e12), 2)}
        log(json.dumps({"chain": line["chain"]}))
    if graph_sparse_ms is not None:
        # the same step with its launches replayed from HIP graphs (no host
        # launch path between kernels): context, not `value`
        line["hip_graph"] = {
            "sparse_ms_per_step": round(graph_sparse_ms, 4),
            "dense_ms_per_step": round(graph_dense_ms, 4),
            "tops": round(float(ops.sum() / (graph_sparse_ms * 1e-3) / 1e12), 2),
            "speedup_vs_dense": round(graph_dense_ms / graph_sparse_ms, 3),
        }
        log(json.dumps({"hip_graph": line["hip_graph"]}))
    if not args.no_mfma_ceiling:
        line["mfma_measured"] = mfma_ceiling(torch)
        log(json.dumps(line["mfma_measured"]))
    if not args.no_secondary and args.config != 2:
        line["deit_base_speedups"] = secondary_workload(2, 3, 2, torch)
        log(json.dumps(line["deit_base_speedups"]))
    if args.copy_calibration:
        # a plain elementwise pass that reads and writes exactly MIB MiB each
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = 4 * n
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
