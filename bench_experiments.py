#!/usr/bin/env python3
"""Experiments around the N:M sparse INT8 GEMM, beside the benchmark line of
bench.py: the planner evaluation in the manner of the paper's Table 1
(--sweep, --sweep-report), the paper's kernel grid of Sec. 6.1
(--paper-grid), the LUT latency predictor of Eq. 1 and the layer-wise search
of Alg. 1 on ViT-L (--predictor), the int8 chaining epilogue (--chaining),
the per-shape roofline table (--shape-report), a DeiT-B layer captured in a
HIP graph (--graph-layer) and the rocprofv3 summary writer
(--rocprof-summary).  Each writes its report under profiles/ when asked and
prints one JSON line.
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

from bench import (PEAK_HBM_GBS, PEAK_INT8_TOPS, PEAK_SPARSE_TOPS, SP42_KINDS, Prepared,  # noqa: E402
                   algorithmic_bytes, default_traffic_path, kernel_source_sha256, log, mfma_ceiling, pattern_name)
from paper_2607_12505_amd import nmspmm  # noqa: E402
from paper_2607_12505_amd import workloads as wl  # noqa: E402


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


def sweep_summary(rows):
    """Table-1 figures of a set of sweep rows: the planner's Top-1 hit rate, its
    average and worst time normalised to the sweep optimum, and the gain over a
    fixed split_k = 1 with the planner's tile."""
    if not rows:
        return None
    norm = np.array([r["t_best_us"] / r["t_planned_us"] for r in rows])
    fixed = np.array([r["t_fixed_split1_us"] / r["t_planned_us"] for r in rows if r["t_fixed_split1_us"]])
    fixed_tile = np.array([r["times"]["0/1"] / r["t_planned_us"] for r in rows if r["times"].get("0/1")])
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
            wname = wl.workload(cfg).name if isinstance(cfg, int) else cfg
            log(f"{wname} {g.name:<20} m={g.m:<6} k={g.k:<5} n={g.n:<5} planned t{chosen[0]}/s{chosen[1]} "
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
          "Command: `python3 bench_experiments.py --predictor --report profiles/predictor_vit_large.md` (repository root).", "",
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
              "Command: `python3 bench_experiments.py --chaining --report profiles/int8_chaining.md` (repository root).  "
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
    torch._int_mm, a measured reference only), int32 output, 50 back-to-back
    runs per window, the fastest of three windows the host queued in time.
    A row whose sparse time differs from the dense GEMM's by more than 3x
    either way is flagged in the report."""
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
              "Command: `python3 bench_experiments.py --paper-grid --report profiles/paper_grid.md` (repository root).  Tokens m in "
              "{64, 128, 256, 512}, n and k in {128, 256, 512, 1024}; 50 % = 2:4 and 4:8, 75 % = 1:4 and 2:8, 87.5 % "
              "= 1:8; int32 output; inputs resident; per call the mean of 50 back-to-back runs between HIP events, "
              "the fastest of three such windows in which the host queued every call before the GPU reached it.  "
              "\"vendor\" = the dense INT8 GEMM of hipBLASLt through torch._int_mm, timed as a reference.  Rows "
              "flagged \"check\" differ from the dense GEMM by more than 3x either way.", "",
              "| sparsity | cases | mean speedup vs this library's dense MFMA GEMM | mean speedup vs the vendor dense GEMM |",
              "|---|---:|---:|---:|"]
        for key, v in summary.items():
            md.append(f"| {key} | {v['cases']} | {v['mean_speedup_vs_own_dense']} | {v['mean_speedup_vs_vendor_dense']} |")
        md += ["", "| m | n | k | pattern | sparse us | dense us | vendor dense us | |",
               "|---:|---:|---:|---|---:|---:|---:|---|"]
        for r in rows:
            odd = not (1 / 3 <= r["dense_us"] / r["sparse_us"] <= 3)
            md.append(f"| {r['m']} | {r['n']} | {r['k']} | {r['pattern']} | {r['sparse_us']} | {r['dense_us']} | "
                      f"{r['vendor_us']} | {'check' if odd else ''} |")
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
            peak = PEAK_SPARSE_TOPS if kind in SP42_KINDS else PEAK_INT8_TOPS
            rate = sp_rate if kind in SP42_KINDS else dn_rate
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
              "Command: `python3 bench_experiments.py --shape-report --report profiles/per_shape_roofline.md` (repository root).  "
              "Every distinct (shape, N:M) of the five workloads; mean of 5 back-to-back launches with inputs resident "
              "(HIP events).  Peaks: HBM 8 TB/s; matrix cores 10.07 dense-equivalent POPS for one 4:2 stream "
              "(smfmac, for 2:4 and the 1:4, 1:8 and 2:8 weights expanded to it), 5.03 POPS for dense and for the mask "
              "layouts expanded to dense tiles.  \"MFMA frac (meas.)\" divides by the rate measured "
              f"in the same run on random int8 operands: smfmac {ceil['smfmac_i32_16x16x128_i8_random_pops']} "
              f"dense-equivalent POPS, dense {ceil['mfma_i32_16x16x64_i8_random_pops']} POPS "
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
          "Commands: `python3 bench_experiments.py --sweep 0,1,2,3,4 --sweep-out sweep.json` (GPU; every (tile, split_k) "
          "candidate timed in two passes of 10 launches each (the second pass in reverse order, each behind a 1 ms "
          "spin), the faster pass kept, outputs rotated over at least two "
          "buffers and at least 512 MB in all, twice the last-level cache), "
          "then `python3 bench_experiments.py --sweep-report sweep.json --report <this file>`.", "",
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
    names = {}
    for r in d["rows"]:
        c = r["cfg"]
        if c not in names:
            names[c] = wl.workload(c).name if isinstance(c, int) else str(c)
        md.append(f"| {names[c]} {r['gemm']} | {r['m']} | {r['k']} | {r['n']} | {r['pattern']} | "
                  f"{r['planned'][0]}/{r['planned'][1]} | {r['t_planned_us']:.1f} | {r['best'][0]}/{r['best'][1]} | "
                  f"{r['t_best_us']:.1f} | {r['t_best_us'] / r['t_planned_us']:.3f} |")
    with open(path, "w") as f:
        f.write("\n".join(md) + "\n")




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

    # the dominant kernel on the dominant GEMM shape: its own grid
    dom_grid = line["roofline"].get("gemm", {}).get("grid")
    sel = _grid_counters(fetch_dir, dom, dom_grid), _grid_counters(write_dir, dom, dom_grid)
    dom_fetch, dom_write = sel if all(sel) else (find(fetch, dom), find(write, dom))
    bytes_per_launch = (np.mean(dom_fetch) * 1024 * f_scale + np.mean(dom_write) * 1024 * w_scale)
    dom_stats = [r for r in stats if dom in r["Name"]][0]
    md = [f"# rocprofv3 summary: `{dom}` on workload `{work}`", ""]
    md += ["Commands (repository root as working directory of the bench; rocprofv3 run from /tmp):", "", "```"]
    md += commands + ["```", ""]
    own = _grid_durations(trace_dir, dom, dom_grid) if dom_grid else None
    gemm = line["roofline"].get("gemm")
    md += [f"Dominant sparse kernel: `{dom}`: {dom_stats['Calls']} calls over every shape of the run, average "
           f"{float(dom_stats['AverageNs']) / 1e3:.2f} us (min {float(dom_stats['MinNs']) / 1e3:.2f}, "
           f"max {float(dom_stats['MaxNs']) / 1e3:.2f})."]
    if own and gemm:
        md += ["", f"On the dominant GEMM shape (m {gemm['m']}, k {gemm['k']}, n {gemm['n']}; patterns "
                   f"{', '.join(gemm['patterns'])}; {dom_grid} workgroups): {len(own)} launches in the trace, average "
                   f"{np.mean(own):.2f} us (median {np.median(own):.2f}); bench.py HIP-event average of the same "
                   f"GEMMs over the timed region ({line['roofline'].get('avg_over_launches', '?')} launches per step "
                   f"without a weight expansion in the call): {line['roofline']['avg_launch_us']:.2f} us."]
    md += [""]
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
    md += launch_shape_table(line, trace_dir, fetch_dir, write_dir, f_scale, w_scale, sq_dir)
    with open(out_md, "w") as f:
        f.write("\n".join(md) + "\n")
    rec = {"kernel": dom, "workload": work, "grid": dom_grid, "bytes_per_launch": int(bytes_per_launch),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "kernel_source_sha256": kernel_source_sha256(), "summary": os.path.basename(out_md)}
    with open(default_traffic_path(work), "w") as f:
        json.dump(rec, f, indent=1)
    print("\n".join(md))




def launch_labels(cfg, carried=True):
    """(kernel name, grid in threads) -> the GEMMs of workload cfg launched that
    way by the planner (sparse leg and dense baseline), from the plans alone.
    carried: the sparse leg was planned with NM_PLAN_EXPAND_CARRIED (bench.py's
    default --expansion tail)."""
    from paper_2607_12505_amd import workloads as wl
    hint = nmspmm.NM_PLAN_EXPAND_CARRIED if carried else 0
    labels = {}
    for g in wl.workload(cfg).gemms:
        # the linear with its batch or stage prefix, without the pattern or the layer index
        short = " ".join(t for t in g.name.split() if ":" not in t and not (t[0] == "L" and t[1:].isdigit()))
        if g.N == g.M:
            plans = [("dense", nmspmm.dense_plan(g.m, g.n, g.k, nmspmm.NM_OUT_I32))]
        else:
            plans = [(f"{g.N}:{g.M}", nmspmm.spmm_plan(nmspmm.compress_size(g.n, g.k, g.N, g.M), g.m,
                                                     nmspmm.NM_OUT_I32 | hint)),
                     ("dense baseline", nmspmm.dense_plan(g.m, g.n, g.k, nmspmm.NM_OUT_I32))]
        for pat, p in plans:
            name = nmspmm.plan_kernel_name(p)
            key = (name, p.grid)
            labels.setdefault(key, set()).add((short, g.m, g.k, g.n, pat))
    return labels


def _workgroups(name, grid_threads):
    if name.startswith("k_gemm_ks"):
        return grid_threads // 256
    parts = [int(x) for x in name[name.index("<") + 1:name.index(">")].split(",")]
    return grid_threads // (64 * parts[1] * parts[2])


def _grid_durations(trace_dir, kernel, grid):
    """Trace durations (us) of `kernel` launched with `grid` workgroups."""
    import csv
    import glob
    out = []
    for r in csv.DictReader(open(glob.glob(os.path.join(trace_dir, "*_kernel_trace.csv"))[0])):
        if kernel in r["Kernel_Name"] and _workgroups(kernel, int(r.get("Grid_Size") or r["Grid_Size_X"])) == grid:
            out.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return out


def _grid_counters(d, kernel, grid):
    """Per-dispatch counter values (summed over a dispatch's rows) of `kernel`
    launched with `grid` workgroups."""
    import csv
    import glob
    if grid is None:
        return None
    per = {}
    for r in csv.DictReader(open(glob.glob(os.path.join(d, "*_counter_collection.csv"))[0])):
        if kernel in r["Kernel_Name"] and _workgroups(kernel, int(r.get("Grid_Size") or r["Grid_Size_X"])) == grid:
            per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    return list(per.values()) or None


def _workload_cfg(line):
    from paper_2607_12505_amd import workloads as wl
    names = {wl.workload(c).name: c for c in range(5)}
    return names.get(line["config"]["workload"])


# Derived columns of the stall-counter table: (title, numerator, denominator,
# scale, format); a column is shown when its counters are present.
_STALL_COLUMNS = (
    ("waiting %", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES", 100.0, "{:.0f}"),
    ("issue-blocked %", "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES", 100.0, "{:.0f}"),
    ("issuing %", "SQ_ACTIVE_INST_ANY", "SQ_WAVE_CYCLES", 100.0, "{:.0f}"),
    ("LDS-issue wait %", "SQ_WAIT_INST_LDS", "SQ_WAVE_CYCLES", 100.0, "{:.1f}"),
    ("MFMA busy %", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", 100.0 * 8 / 1024, "{:.1f}"),
    ("LDS conflict %", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", 100.0, "{:.2f}"),
    ("LDS data FIFO full %", "SQ_LDS_DATA_FIFO_FULL", "SQ_LDS_IDX_ACTIVE", 100.0, "{:.1f}"),
    ("L2 read latency (cycles)", "TCP_TCC_READ_REQ_LATENCY_sum", "TCP_TCC_READ_REQ_sum", 1.0, "{:.0f}"),
)


def pmc_stall_table(dirs, cfg, commands, out_md):
    """Per launch shape (kernel and grid) of workload cfg: per-dispatch means of
    the counters found in the rocprofv3 counter-collection CSVs of `dirs` (one
    directory per --pmc pass of the same bench run), as the ratios of
    _STALL_COLUMNS.  Wave-cycle counters are summed over all waves, so their
    ratios are fractions of the waves' resident time."""
    import csv
    import glob
    import re
    per = {}
    for d in dirs:
        for r in csv.DictReader(open(glob.glob(os.path.join(d, "*_counter_collection.csv"))[0])):
            m = re.search(r"(k_gemm(?:_ks)?<[^>]*>)", r["Kernel_Name"])
            if not m:
                continue
            k = m.group(1)
            key = (k, _workgroups(k, int(r["Grid_Size"])))
            disp = per.setdefault(key, {}).setdefault(r["Counter_Name"], {})
            tag = (d, r["Dispatch_Id"])
            disp[tag] = disp.get(tag, 0.0) + float(r["Counter_Value"])
    labels = launch_labels(cfg)
    from paper_2607_12505_amd import workloads as wl
    cols = [c for c in _STALL_COLUMNS if any(c[1] in v and c[2] in v for v in per.values())]
    md = [f"# rocprofv3 stall counters per launch shape: workload `{wl.workload(cfg).name}`", "",
          "Commands (repository root as working directory of the bench; rocprofv3 run from /tmp):", "", "```"]
    md += list(commands) + ["```", "",
                            "Per dispatch means; the wave-cycle counters (SQ_WAVE_CYCLES, SQ_WAIT_ANY, SQ_WAIT_INST_ANY, "
                            "SQ_ACTIVE_INST_ANY, SQ_WAIT_INST_LDS) are summed over every resident wave, so their ratios "
                            "are shares of the waves' resident time: *waiting* = at an s_waitcnt or barrier, "
                            "*issue-blocked* = ready but its functional unit (mostly the matrix core) busy, *issuing* = "
                            "issuing an instruction.  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x "
                            "1024 SIMDs); LDS ratios per LDS-active cycle; L2 read latency = TCP_TCC_READ_REQ_LATENCY / "
                            "TCP_TCC_READ_REQ (cycles from the CU's L1 to L2 and back, per request).", "",
          "| kernel | workgroups | GEMMs | dispatches | " + " | ".join(c[0] for c in cols) + " |",
          "|---|---:|---|---:|" + "---:|" * len(cols)]
    rows = []
    for key, cs in per.items():
        if not cols or not all(c[1] in cs and c[2] in cs for c in cols[:1]):
            continue
        gemms = labels.get(key)
        what = (", ".join(sorted({f"{g[0]} {g[4]}" for g in gemms})) if gemms else
                "a launch with workgroups beyond the planned grid (a GEMM carrying an expansion)")
        if gemms and len({g[1:4] for g in gemms}) == 1:
            _, m, k, n, _ = sorted(gemms)[0]
            what += f" (m {m}, k {k}, n {n})"
        vals = []
        for _, num, den, scale, fmt in cols:
            if num in cs and den in cs:
                a, b = np.mean(list(cs[num].values())), np.mean(list(cs[den].values()))
                vals.append(fmt.format(scale * a / b) if b else "")
            else:
                vals.append("")
        nd = len(cs[cols[0][2]])   # dispatches of the pass that holds the first column's counters
        rows.append((-nd, f"| `{key[0]}` | {key[1]} | {what} | {nd} | " + " | ".join(vals) + " |"))
    md += [r for _, r in sorted(rows)]
    with open(out_md, "w") as f:
        f.write("\n".join(md) + "\n")
    print("\n".join(md))


def launch_shape_table(line, trace_dir, fetch_dir, write_dir, f_scale, w_scale, sq_dir):
    """Per launch shape (kernel and grid) of the workload: average duration from
    the kernel trace, scaled HBM bytes per dispatch, the algorithmic bytes and
    ops of the GEMMs launched that way, the achieved fraction of the HBM and
    matrix-instruction peaks, and matrix-core busy time."""
    import csv
    import glob
    import re
    cfg = _workload_cfg(line)
    if cfg is None:
        return []
    labels = launch_labels(cfg, carried=str(line.get("compact_weight_expansion", "")).startswith("carried"))
    work = wl.workload(cfg)

    def short(n):
        m = re.search(r"(k_gemm(?:_ks)?<[^>]*>)", n)
        return m.group(1) if m else None

    durs = {}
    for r in csv.DictReader(open(glob.glob(os.path.join(trace_dir, "*_kernel_trace.csv"))[0])):
        k = short(r["Kernel_Name"])
        if k:
            key = (k, _workgroups(k, int(r.get("Grid_Size") or r["Grid_Size_X"])))
            durs.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)

    def per_shape(d, counter=None):
        out = {}
        for r in csv.DictReader(open(glob.glob(os.path.join(d, "*_counter_collection.csv"))[0])):
            k = short(r["Kernel_Name"])
            if not k or (counter and r["Counter_Name"] != counter):
                continue
            key = (k, _workgroups(k, int(r["Grid_Size"])), int(r["Dispatch_Id"]))
            out[key] = out.get(key, 0.0) + float(r["Counter_Value"])
        agg = {}
        for (k, g, _), v in out.items():
            agg.setdefault((k, g), []).append(v)
        return agg

    fetch, write = per_shape(fetch_dir), per_shape(write_dir)
    busy = per_shape(sq_dir, "SQ_VALU_MFMA_BUSY_CYCLES") if sq_dir else {}
    active = per_shape(sq_dir, "GRBM_GUI_ACTIVE") if sq_dir else {}
    md = ["", "Per launch shape of the workload (kernel and grid, matched to the GEMMs the planner launches that "
          "way): average duration from the kernel trace, HBM bytes per dispatch from the scaled counters, "
          "algorithmic bytes (X + stored weight + the workload's outputs: int32 Y, and fp16 Yh with its scales "
          "where the workload writes it) and dense-equivalent ops of those GEMMs, and the "
          "fraction of the HBM peak (8 TB/s) and of the matrix-instruction peak of the kind (2:4-operand "
          "kernels against 10.07 dense-equivalent POPS, dense against 5.03):", "",
          "| kernel | workgroups | GEMMs | us | HBM MB | alg. MB | HBM frac | POPS | MFMA frac | MFMA busy % |",
          "|---|---:|---|---:|---:|---:|---:|---:|---:|---:|"]
    rows = []
    for (name, grid), gemms in labels.items():
        key = (name, grid)
        if key not in durs:
            continue
        us = float(np.mean(durs[key]))
        if len({g[1:4] for g in gemms}) > 1:
            # GEMMs of different shapes launched alike (same kernel, same grid):
            # the trace cannot tell their launches apart
            what = ", ".join(sorted({f"{s} {p} (m {m}, k {k}, n {n})" for s, m, k, n, p in gemms}))
            rows.append((0.0, f"| `{name}` | {grid} | {what}: shapes not separable in the trace | {us:.1f} (mixed) "
                              "| | | | | | |"))
            continue
        _, m, k, n, _ = sorted(gemms)[0]

        def stored(pat):
            if pat.startswith("dense"):
                return n * k
            d = nmspmm.compress_size(n, k, *(int(x) for x in pat.split(":")))
            return d.vals_bytes + d.meta_bytes

        # the GEMMs of one launch shape share m, k and n; their stored weights
        # differ by pattern (a small part of the bytes): averaged
        alg = (m * k + (4 * m * n if work.out_int32 else 0) + (2 * m * n + 4 * n if work.out_f16 else 0)
               + float(np.mean([stored(p) for *_, p in gemms])))
        ops = 2.0 * m * n * k
        hbm = ((np.mean(fetch[key]) * 1024 * f_scale + np.mean(write[key]) * 1024 * w_scale) / 1e6
               if key in fetch and key in write else float("nan"))
        peak = 5.03 if name.startswith("k_gemm<3") or name.startswith("k_gemm_ks<3") else 10.07
        pops = ops / (us * 1e-6) / 1e15
        mb = (100.0 * np.mean(busy[key]) / (np.mean(active[key]) / 8 * 1024)
              if key in busy and key in active else float("nan"))
        what = ", ".join(sorted({f"{s} {p}" for s, _, _, _, p in gemms}))
        rows.append((-us, f"| `{name}` | {grid} | {what} (m {m}, k {k}, n {n}) | {us:.1f} | {hbm:.1f} | "
                          f"{alg / 1e6:.1f} | {alg / (us * 1e-6) / 8e12:.3f} | {pops:.3f} | {pops / peak:.3f} | "
                          f"{mb:.1f} |"))
    md += [r for _, r in sorted(rows)]
    return md


def chain_sweep(torch, cfg, rounds, out_path, report, carried=False):
    """Planner evaluation inside a workload's own steps: for every distinct
    (shape, kind) of the sparse leg, every (tile, expansion) candidate with
    split_k = 1 is put on all GEMMs of that key and timed in ABBA rounds of
    whole steps (sparse leg, dense leg) with an event after every GEMM, so each
    candidate sees the cache state of the step itself (every layer with its
    own cold inputs and outputs in the ViT-L chain).  Reports per key the
    planner's choice, the fastest candidate and their times.

    carried: the steps run as bench.py's default does (expansions carried by
    the previous launch, plans with NM_PLAN_EXPAND_CARRIED); a candidate's
    time then also counts the launches that carry its expansions."""
    import bench
    work, preps = bench.prepare(cfg, torch)
    if carried:
        bench.carry_expansions(preps)
    sp = [p.run_sparse for p in preps]
    dn = [p.run_dense for p in preps]
    bench.abba(torch, sp, dn, 1, per_call=True)
    keys = {}
    for i, p in enumerate(preps):
        keys.setdefault((p.g.m, p.g.k, p.g.n, p.sparse_kind()), []).append(i)
    rows = []
    # the dense leg too (the baseline of every shape), keyed like a dense kind
    for i, p in enumerate(preps):
        keys.setdefault((p.g.m, p.g.k, p.g.n, "baseline"), []).append(i)
    for (m, k, n, kind), idx in sorted(keys.items(), key=lambda kv: (kv[0][:3], str(kv[0][3]))):
        first = preps[idx[0]]
        baseline = kind == "baseline"
        planned = nmspmm.NmPlan.from_buffer_copy(first.dplan if baseline else first.splan)
        compact = not baseline and kind not in (nmspmm.NM_KIND_SP42, nmspmm.NM_KIND_DENSE)
        times = {}
        ref = {}   # carried: per-call times under the first in-kernel-expansion candidate
        for tile in range(nmspmm.num_tiles()):
            for expand in ((0, 1) if compact else (0,)):
                cand = nmspmm.make_plan(nmspmm.NM_KIND_DENSE if baseline else kind, tile, 1, expand)
                try:
                    if baseline or kind == nmspmm.NM_KIND_DENSE:
                        cand.tile_n, cand.tile_m = nmspmm.tile_info(tile)
                    else:
                        cand = nmspmm.spmm_plan_complete(first.packed.desc, m, cand)
                except nmspmm.NmError:
                    continue
                for i in idx:
                    preps[i].set_dense_plan(cand) if baseline else preps[i].set_sparse_plan(cand)
                if carried:
                    bench.relink_carried(preps)
                try:
                    ta, tb = bench.abba(torch, sp, dn, rounds, per_call=True)
                except nmspmm.NmError:
                    continue
                if carried and not baseline:
                    # per GEMM of the key: its own time, plus what carrying its
                    # expansion adds to the launch before it (that launch's time
                    # here minus its time under an in-kernel-expansion candidate)
                    pc = ta.mean(axis=0) * 1e3
                    carriers = [i - 1 for i in idx
                                if i > 0 and i - 1 not in idx and preps[i - 1].tail_next is preps[i]]
                    if expand == 0:
                        ref.setdefault("pc", pc)
                    if carriers and "pc" not in ref:
                        continue
                    extra = sum(pc[j] - ref["pc"][j] for j in carriers)
                    times[(tile, expand)] = float(pc[idx].sum() + extra) / len(idx)
                else:
                    times[(tile, expand)] = float((tb if baseline else ta)[:, idx].mean()) * 1e3
        for i in idx:
            preps[i].set_dense_plan(planned) if baseline else preps[i].set_sparse_plan(planned)
        if carried:
            bench.relink_carried(preps)
        best = min(times, key=times.get)
        t_plan = times.get((planned.tile, planned.expand))
        row = {"m": m, "k": k, "n": n, "kind": kind, "gemms": len(idx), "planned": [planned.tile, planned.expand],
               "best": list(best), "t_planned_us": t_plan, "t_best_us": times[best],
               "times": {f"{t}/{e}": round(v, 2) for (t, e), v in sorted(times.items())}}
        rows.append(row)
        log(f"m={m} k={k} n={n} kind {kind} ({len(idx)} GEMMs): planned t{planned.tile}/e{planned.expand} "
            f"{t_plan:.1f} us, best t{best[0]}/e{best[1]} {times[best]:.1f} us")
    summary = {"workload": work.name, "cases": len(rows),
               "top1_hit_rate": round(float(np.mean([r["planned"] == r["best"] for r in rows])), 3),
               "avg_norm_perf": round(float(np.mean([r["t_best_us"] / r["t_planned_us"] for r in rows])), 3),
               "worst_norm_perf": round(float(min(r["t_best_us"] / r["t_planned_us"] for r in rows)), 3)}
    if out_path:
        with open(out_path, "w") as f:
            json.dump({"summary": summary, "rows": rows}, f)
    if report:
        flag = " --carried" if carried else ""
        md = [f"# Planner choices inside the {work.name} steps" + (" with carried expansions" if carried else ""), "",
              f"Command: `python3 bench_experiments.py --chain-sweep {cfg}{flag} --rounds {rounds} --report {report}` (repository root).  "
              "For every distinct (shape, kind) of the sparse leg, every tile with split_k = 1 (and, for the compact "
              "kinds, both places of the weight expansion: e0 inside every workgroup, e1 once per call) is put on "
              "all GEMMs of that key and timed inside whole steps (ABBA rounds of the sparse and dense legs, an "
              f"event after every GEMM, {rounds} rounds); times are means per GEMM in microseconds.  Kinds: "
              "1 = 2:4, 2 = 1:4, 3 = dense, 4 = 1:8, 5 = 2:8, 6-8 = 3:8-5:8; \"baseline\": the dense leg (the "
              "dense INT8 GEMM every speedup divides by) of that shape." +
              (("  Expansions once per call are carried by the previous GEMM's launch, as bench.py runs the steps; a "
                "compact kind's time per GEMM includes the share of those launches (the planned choice is "
                "NM_PLAN_EXPAND_CARRIED's).") if carried else ""), "",
              f"Top-1 hit rate {summary['top1_hit_rate']}, average normalised performance "
              f"{summary['avg_norm_perf']}, worst {summary['worst_norm_perf']}.", "",
              "| m | k | n | kind | GEMMs | planned | us | best | us | ratio | all candidates (tile/expand: us) |",
              "|---:|---:|---:|---:|---:|---|---:|---|---:|---:|---|"]
        for r in rows:
            cands = ", ".join(f"{c}: {v}" for c, v in r["times"].items())
            md.append(f"| {r['m']} | {r['k']} | {r['n']} | {r['kind']} | {r['gemms']} | {r['planned'][0]}/"
                      f"{r['planned'][1]} | {r['t_planned_us']:.1f} | {r['best'][0]}/{r['best'][1]} | "
                      f"{r['t_best_us']:.1f} | {r['t_best_us'] / r['t_planned_us']:.3f} | {cands} |")
        with open(report, "w") as f:
            f.write("\n".join(md) + "\n")
    return summary


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--sweep", type=str, default=None,
                    help="planner evaluation over the given comma-separated configs (e.g. 0,1,2,3,4); 'grid' adds "
                         "the paper's kernel grid")
    ap.add_argument("--sweep-out", type=str, default=None, help="JSON file for the sweep results")
    ap.add_argument("--sweep-report", type=str, default=None, metavar="SWEEP_JSON",
                    help="markdown report (--report) of a sweep JSON (no GPU needed)")
    ap.add_argument("--rocprof-summary", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"), default=None,
                    help="summarise rocprofv3 CSV output of a bench run (no GPU needed)")
    ap.add_argument("--bench-json", type=str, default=None, help="bench output line used by --rocprof-summary")
    ap.add_argument("--rocprof-sq", type=str, default=None,
                    help="rocprofv3 counter output with MFMA busy / LDS bank conflict counters (--rocprof-summary)")
    ap.add_argument("--pmc-stalls", nargs="+", metavar="PASS_DIR", default=None,
                    help="per-launch-shape table of stall counters from rocprofv3 --pmc passes of one bench run "
                         "(no GPU needed; with --summary-out, --commands, --stall-config)")
    ap.add_argument("--stall-config", type=int, default=4, help="workload of the --pmc-stalls bench run")
    ap.add_argument("--carried", action="store_true",
                    help="--chain-sweep with the expansions carried by the previous launch (bench.py's default)")
    ap.add_argument("--summary-out", type=str, default=None, help="markdown file written by --rocprof-summary")
    ap.add_argument("--commands", type=str, default=None, help="file with the profiling commands to quote")
    ap.add_argument("--copy-calibration", type=int, default=256, metavar="MIB",
                    help="size of the calibration copy the bench run made (--rocprof-summary)")
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
    ap.add_argument("--chain-sweep", type=int, default=None, metavar="CFG",
                    help="tile and expansion candidates timed inside the steps of workload CFG (e.g. 4)")
    ap.add_argument("--rounds", type=int, default=2, help="ABBA rounds per candidate of --chain-sweep")
    ap.add_argument("--cal", type=int, default=64, help="calibration configurations for --predictor")
    ap.add_argument("--test", type=int, default=32, help="random test configurations for --predictor")
    ap.add_argument("--report", type=str, default=None, help="markdown report of an experiment")
    args = ap.parse_args()

    if args.sweep_report:
        write_sweep_report(args.sweep_report, args.report)
        return
    if args.pmc_stalls:
        cmds = open(args.commands).read().strip().splitlines() if args.commands else []
        pmc_stall_table(args.pmc_stalls, args.stall_config, cmds, args.summary_out)
        return
    if args.rocprof_summary:
        cmds = open(args.commands).read().strip().splitlines() if args.commands else []
        rocprof_summary(*args.rocprof_summary, args.bench_json, args.copy_calibration, cmds, args.summary_out,
                        args.rocprof_sq)
        return

    import torch
    if not torch.cuda.is_available():
        print("bench_experiments.py needs a GPU for this experiment", file=sys.stderr)
        sys.exit(1)
    nmspmm.lib()
    torch.cuda.set_device(0)
    if args.chain_sweep is not None:
        print(json.dumps({"chain_sweep": chain_sweep(torch, args.chain_sweep, args.rounds, args.sweep_out,
                                                     args.report, carried=args.carried)}), flush=True)
    elif args.sweep:
        summary = sweep([c if c == "grid" else int(c) for c in args.sweep.split(",")], torch, 10, args.sweep_out)
        print(json.dumps({"planner_evaluation": summary}), flush=True)
    elif args.chaining:
        print(json.dumps({"chaining": chaining_experiment(torch, args.report)}), flush=True)
    elif args.paper_grid:
        print(json.dumps({"paper_grid": paper_grid(torch, args.report)}), flush=True)
    elif args.predictor:
        print(json.dumps({"predictor": predictor_experiment(torch, args.cal, args.test, args.report)}), flush=True)
    elif args.shape_report:
        print(json.dumps({"shape_report": shape_report(torch, args.report)}), flush=True)
    elif args.graph_layer:
        print(json.dumps({"graph_layer": graph_layer(torch)}), flush=True)
    else:
        ap.print_help(sys.stderr)
        sys.exit(2)


if __name__ == "__main__":
    main()
