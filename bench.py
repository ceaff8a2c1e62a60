#!/usr/bin/env python3
"""Benchmark of the N:M sparse INT8 GEMM on one MI355X.

Metric: dense-equivalent INT8 TOPS (2 m n k / t) of the sparse GEMMs of a ViT
workload, and their speedup over the dense INT8 MFMA GEMM of the same shapes.

Default workload: the 96 linears of ViT-Large/16 at 384 px, batch 32
(m = 18464 tokens, hidden 1024, MLP 4096), each with its seeded layer-wise
N:M pattern from {dense, 4:8, 2:4, 2:8, 1:4}, run in network order.  One step
= one pass over every linear of the workload with the sparse kernels
(nm_spmm on the packed weights; the dense layers of the draw run the dense
kernel).  Inputs are resident in HBM before timing starts; packing is
offline and untimed (the paper times inference only, Sec. 6.1).

* The timed region: W untimed steps, then exactly K steps between two device
  synchronisations; `value` = dense-equivalent ops per step / wall time per
  step (`ms_per_step`).
* The speedup over the dense baseline (nm_gemm_i8_dense on the same weights
  stored densely) comes from whole steps of both legs in ABBA order (sparse,
  dense, dense, sparse; one event pair per leg), so a bias from a leg's
  position cancels; beside it the same protocol runs the dense leg against
  itself (an A/A control whose ratio shows the measurement's own spread).
* Per pattern and per kernel: ABBA rounds with an event after every GEMM.
* `roofline`: the dominant sparse kernel (most time per step) against the
  roofline that binds it, from its HIP-event launch times.

Prints one JSON line on stdout; human-readable tables go to stderr.
"""
from __future__ import annotations

import argparse
import gc
import ctypes
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
# kernel families on the structured-sparse instruction (the others run the dense one)
SP42_KINDS = (nmspmm.NM_KIND_SP42, nmspmm.NM_KIND_C14, nmspmm.NM_KIND_C18, nmspmm.NM_KIND_C28)
KERNEL_SOURCE = os.path.join(ROOT, "paper_2607_12505_amd", "csrc", "nmspmm_kernels.hip")


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
    arguments for both the sparse call and the dense baseline.

    A compact weight whose plan expands it once per call (expand = 1) is,
    when side_stream is set, expanded by nm_expand on that stream into a
    buffer of its own, and the GEMM on the main stream waits for it: the
    expansion of a layer then runs while earlier GEMMs are still running,
    instead of between two GEMMs.  The expansion waits for the previous GEMM
    that read its buffer."""

    side_stream = None

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
        self._torch = torch
        # dense baseline
        self.dplan = nmspmm.dense_plan(g.m, g.n, g.k, out)
        self.dense_fn = nmspmm.lib().nm_gemm_i8_dense_ex
        if self.sparse_kernel:
            self.packed = nmspmm.compress(W, g.N, g.M)
            self.dw = nmspmm.DeviceWeight.from_packed(self.packed)
            self.splan = nmspmm.spmm_plan(self.packed.desc, g.m, out)
            self.sparse_fn = nmspmm.lib().nm_spmm_ex
        else:
            # a dense layer inside a layer-wise chain runs the dense kernel on both sides
            self.splan = nmspmm.NmPlan.from_buffer_copy(self.dplan)
            self.sparse_fn = nmspmm.lib().nm_gemm_i8_dense_ex
        self.sws = self.dws = self.ews = self.exp_buf = None
        self.ahead = False
        self.pre_expanded = False     # the weight is expanded by the previous GEMM's launch (tail mode)
        self.tail_next = None         # the next GEMM, whose weight this launch expands (tail mode)
        self._build_args()

    def _workspace(self, plan, old):
        need = max(nmspmm.workspace_size(plan, self.g.m, self.g.n), 16)
        if old is not None and old.numel() >= need:
            return old
        return self._torch.zeros(need, dtype=self._torch.uint8, device="cuda")

    def _build_args(self):
        """ctypes arguments of both calls for the current plans."""
        g = self.g
        ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        stream = ctypes.c_void_p(self._torch.cuda.current_stream().cuda_stream)
        self.dws = self._workspace(self.dplan, self.dws)
        self.dense_args = (ptr(self.Xd), g.m, ptr(self.Wd), g.n, g.k, ptr(self.Yd), ptr(self.scale),
                           ptr(self.Yhd), ptr(self.dws), self.dws.numel(), stream, ctypes.byref(self.dplan))
        self.sws = self._workspace(self.splan, self.sws)
        if self.sparse_kernel:
            self.sparse_args = (ptr(self.Xd), g.m, ptr(self.dw.vals), ptr(self.dw.meta),
                                ctypes.byref(self.packed.desc), ptr(self.Y), ptr(self.scale), ptr(self.Yh),
                                ptr(self.sws), self.sws.numel(), stream, ctypes.byref(self.splan))
        else:
            self.sparse_args = (ptr(self.Xd), g.m, ptr(self.Wd), g.n, g.k, ptr(self.Y), ptr(self.scale),
                                ptr(self.Yh), ptr(self.sws), self.sws.numel(), stream, ctypes.byref(self.splan))
        self.ahead = bool(self.sparse_kernel and self.splan.expand and Prepared.side_stream is not None)
        if self.ahead:
            torch = self._torch
            e, nbytes = nmspmm.expand_size(self.packed.desc)
            if self.exp_buf is None or self.exp_buf.numel() < nbytes:
                self.exp_buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
            self.edesc = e
            # the plan of the GEMM on the expanded weight: the same tile and split
            self.eplan = nmspmm.spmm_plan_complete(e, g.m, nmspmm.make_plan(e.kind, self.splan.tile,
                                                                            self.splan.split_k, 0))
            self.ews = self._workspace(self.eplan, self.ews)
            side = ctypes.c_void_p(Prepared.side_stream.cuda_stream)
            vals = self.exp_buf.data_ptr()
            meta = ctypes.c_void_p(vals + e.vals_bytes) if e.meta_bytes else None
            self.expand_args = (ctypes.byref(self.packed.desc), ptr(self.dw.vals), ptr(self.dw.meta),
                                ptr(self.exp_buf), self.exp_buf.numel(), side)
            self.ahead_args = (ptr(self.Xd), g.m, ctypes.c_void_p(vals), meta, ctypes.byref(self.edesc), ptr(self.Y),
                               ptr(self.scale), ptr(self.Yh), ptr(self.ews), self.ews.numel(), stream,
                               ctypes.byref(self.eplan))
            self.ev_expanded = torch.cuda.Event()
            self.ev_used = torch.cuda.Event()
            self.main_stream = torch.cuda.current_stream()

    def _build_expanded(self):
        """Buffer, descriptor, plan and ctypes arguments of the GEMM on this
        layer's expanded weight (the same tile and split as its plan)."""
        torch = self._torch
        g = self.g
        ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        e, nbytes = nmspmm.expand_size(self.packed.desc)
        if self.exp_buf is None or self.exp_buf.numel() < nbytes:
            self.exp_buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.edesc = e
        self.eplan = nmspmm.spmm_plan_complete(e, g.m, nmspmm.make_plan(e.kind, self.splan.tile, self.splan.split_k, 0))
        self.ews = self._workspace(self.eplan, self.ews)
        vals = self.exp_buf.data_ptr()
        meta = ctypes.c_void_p(vals + e.vals_bytes) if e.meta_bytes else None
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        self.pre_args = (ptr(self.Xd), g.m, ctypes.c_void_p(vals), meta, ctypes.byref(self.edesc), ptr(self.Y),
                         ptr(self.scale), ptr(self.Yh), ptr(self.ews), self.ews.numel(), stream,
                         ctypes.byref(self.eplan))

    def carry_expansion_of(self, nxt):
        """Tail mode: this GEMM's launch also expands the weight of `nxt` (a
        GEMM whose plan expands its compact weight once per call), which then
        runs on the expanded weight with no expansion launch of its own."""
        nxt.pre_expanded = True
        nxt._build_expanded()
        self.tail_next = nxt
        self.job = nmspmm.NmExpandJob(ctypes.pointer(nxt.packed.desc), nxt.dw.vals.data_ptr(),
                                      nxt.dw.meta.data_ptr(), nxt.exp_buf.data_ptr(), nxt.exp_buf.numel())
        self.outs = nmspmm.NmOutputs(self.Y.data_ptr() if self.Y is not None else None,
                                     self.Yh.data_ptr() if self.Yh is not None else None,
                                     self.scale.data_ptr(), None, None)
        a = self.sparse_args
        if self.pre_expanded:
            a = self.pre_args
        if self.sparse_kernel:
            # (X, m, vals, meta, desc, out, ws, ws_bytes, stream, plan, job)
            self.tail_fn = nmspmm.lib().nm_spmm_out_expand
            self.tail_args = (a[0], a[1], a[2], a[3], a[4], ctypes.byref(self.outs), a[8], a[9], a[10], a[11],
                              ctypes.byref(self.job))
        else:
            self.tail_fn = nmspmm.lib().nm_gemm_i8_dense_out_expand
            self.tail_args = (a[0], a[1], a[2], a[3], a[4], ctypes.byref(self.outs), a[8], a[9], a[10], a[11],
                              ctypes.byref(self.job))

    def set_sparse_plan(self, plan):
        """Runs the sparse-leg call with `plan` from now on (a completed plan
        of this GEMM's kind); the workspace grows as the plan needs."""
        self.splan = nmspmm.NmPlan.from_buffer_copy(plan)
        self._build_args()

    def set_dense_plan(self, plan):
        """Runs the dense-baseline call with `plan` from now on."""
        self.dplan = nmspmm.NmPlan.from_buffer_copy(plan)
        self._build_args()

    def sparse_kind(self):
        return self.packed.desc.kind if self.sparse_kernel else nmspmm.NM_KIND_DENSE

    def kernel_name(self, plan):
        return nmspmm.plan_kernel_name(plan)

    def expands_in_call(self):
        """Whether the sparse call launches an expansion (a kernel before its
        GEMM, or workgroups appended to it)."""
        own = self.sparse_kernel and self.splan.expand and not self.ahead and not self.pre_expanded
        return bool(own or self.tail_next is not None)

    def run_sparse(self):
        if self.tail_next is not None:
            st = self.tail_fn(*self.tail_args)
        elif self.pre_expanded:
            st = nmspmm.lib().nm_spmm_ex(*self.pre_args)
        elif self.ahead:
            side = Prepared.side_stream
            side.wait_event(self.ev_used)
            st = nmspmm.lib().nm_expand(*self.expand_args)
            if st:
                raise nmspmm.NmError(st, f"expand {self.g.name}")
            self.ev_expanded.record(side)
            self.main_stream.wait_event(self.ev_expanded)
            st = nmspmm.lib().nm_spmm_ex(*self.ahead_args)
            self.ev_used.record(self.main_stream)
        else:
            st = self.sparse_fn(*self.sparse_args)
        if st:
            raise nmspmm.NmError(st, f"sparse {self.g.name}")

    def run_dense(self):
        st = self.dense_fn(*self.dense_args)
        if st:
            raise nmspmm.NmError(st, f"dense {self.g.name}")


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
    ev = [(timing_event(), timing_event()) for _ in range(reps)]
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




# ---------------------------------------------------------------------------
# timing

def timing_event():
    """An event for the timings below, recorded without the system-scope fence
    of a default HIP event (whose cache write-back and invalidation would add
    microseconds after every timed GEMM and hand the next one cold caches)."""
    return nmprobe.TimingEvent()


def sleep_cycles_for(launches: int) -> int:
    """Device-side sleep before a batch of `launches` host-side queue
    operations (kernel launches and event records), long enough for the host
    to queue them ahead of the GPU (about 15 us each, at most 20 ms), so host
    launch overhead stays out of the event times."""
    return int(2.1e9 * min(15e-6 * launches, 20e-3))


def hold_side_stream(torch):
    """The side stream's next work waits for everything issued so far on the
    current stream (so expansions of a leg cannot run during an earlier,
    untimed leg or sleep)."""
    if Prepared.side_stream is not None:
        ev = torch.cuda.Event()
        ev.record()
        Prepared.side_stream.wait_event(ev)


class _NoGC:
    """Python's garbage collector paused while the host queues timed work: a
    collection pause longer than the device sleep that gives the host its head
    start would otherwise land inside an event interval."""

    def __enter__(self):
        self.was = gc.isenabled()
        gc.disable()

    def __exit__(self, *exc):
        if self.was:
            gc.enable()


def timed_steps(preps, steps, torch):
    """The contract's timed region: `steps` steps of the sparse leg back to
    back between two synchronisations.  Returns (wall ms per step, event ms of
    each step)."""
    with _NoGC():
        return _timed_steps(preps, steps, torch)


def _timed_steps(preps, steps, torch):
    ev = [(timing_event(), timing_event()) for _ in range(steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record()
        hold_side_stream(torch)
        for p in preps:
            p.run_sparse()
        e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    return wall * 1e3 / steps, np.array([e0.elapsed_time(e1) for e0, e1 in ev])


def abba(torch, calls_a, calls_b, rounds, per_call=False):
    """Legs A and B (lists of launch callables) in ABBA order, `rounds` times,
    each round behind a device sleep and an untimed leg of B (so the first
    timed leg does not start from the clock and cache state the sleep
    leaves).  Returns the times of A and of B: one value per leg
    ([2 * rounds]) or, with per_call, one per call ([2 * rounds,
    len(calls)]), in ms."""
    with _NoGC():
        return _abba(torch, calls_a, calls_b, rounds, per_call)


def _abba(torch, calls_a, calls_b, rounds, per_call):
    recs = []
    # a round queues an untimed leg and four timed legs, with an event after
    # every call in per-call mode: the sleep covers all of it, so that the
    # GPU never waits for the host inside a timed leg (a short GEMM's event
    # time would otherwise include that wait)
    ops = 5 * max(len(calls_a), len(calls_b)) * (2 if per_call else 1) + 8
    for _ in range(rounds):
        torch.cuda._sleep(sleep_cycles_for(ops))
        for c in calls_b:
            c()
        for which in (0, 1, 1, 0):
            ev = [timing_event()]
            ev[0].record()
            hold_side_stream(torch)
            for c in (calls_a if which == 0 else calls_b):
                c()
                if per_call:
                    ev.append(timing_event())
                    ev[-1].record()
            if not per_call:
                ev.append(timing_event())
                ev[-1].record()
            recs.append((which, ev))
    torch.cuda.synchronize()
    out = ([], [])
    for which, ev in recs:
        t = [ev[i].elapsed_time(ev[i + 1]) for i in range(len(ev) - 1)]
        out[which].append(t if per_call else t[0])
    return np.array(out[0]), np.array(out[1])


def ratio_stats(ta, tb):
    """Σ tb / Σ ta, and the spread of the per-round ratios (a round = its two
    legs of each side)."""
    ra = ta.reshape(-1, 2).sum(axis=1)
    rb = tb.reshape(-1, 2).sum(axis=1)
    per_round = rb / ra
    return {"ratio": round(float(tb.sum() / ta.sum()), 4),
            "round_min": round(float(per_round.min()), 4), "round_max": round(float(per_round.max()), 4),
            "round_std": round(float(per_round.std()), 4), "rounds": int(per_round.size)}


def per_key_speedups(preps, ts, td, keyfn):
    """TOPS and speedup per key from per-GEMM mean times (ms)."""
    out = {}
    for key in sorted({keyfn(p) for p in preps}, key=str):
        sel = [i for i, p in enumerate(preps) if keyfn(p) == key]
        ops = sum(preps[i].g.dense_eq_ops for i in sel)
        s, d = ts[sel].sum(), td[sel].sum()
        out[key] = {"tops": round(float(ops / (s * 1e-3) / 1e12), 1), "speedup_vs_dense": round(float(d / s), 3)}
    return out


def prepare(cfg, torch):
    work = wl.workload(cfg)
    xd, xh = {}, {}
    # a chain workload gives every linear its own input and output (as a
    # network's layers have), so every operand and output is cold
    preps = [Prepared(cfg, g, xd, xh if not work.chain else None, work.out_int32, work.out_f16, torch,
                      use_dense_kernel=(g.N == g.M)) for g in work.gemms]
    torch.cuda.synchronize()
    return work, preps


def carry_expansions(preps):
    """Tail mode over a sequence of GEMMs: the compact weights are planned for
    carried expansions (NM_PLAN_EXPAND_CARRIED), and every GEMM whose plan
    expands its weight once per call, except the first of the sequence, has
    that expansion carried by the launch of the GEMM before it."""
    for i, p in enumerate(preps):
        # the first GEMM of the sequence has no launch before it to carry its expansion
        if i > 0 and p.sparse_kernel and p.packed.desc.kind not in (nmspmm.NM_KIND_SP42, nmspmm.NM_KIND_DENSE):
            mode = (nmspmm.NM_OUT_I32 if p.out_i32 else 0) | (nmspmm.NM_OUT_F16 if p.out_f16 else 0)
            p.set_sparse_plan(nmspmm.spmm_plan(p.packed.desc, p.g.m, mode | nmspmm.NM_PLAN_EXPAND_CARRIED))
    relink_carried(preps)


def relink_carried(preps):
    """Re-derives which launch carries which expansion from the current plans
    (after plans changed)."""
    for p in preps:
        p.tail_next = None
        p.pre_expanded = False
        p._build_args()
    for prev, nxt in zip(preps, preps[1:]):
        if nxt.sparse_kernel and nxt.splan.expand and prev.tail_next is None:
            prev.carry_expansion_of(nxt)


def secondary_workload(cfg, rounds, torch, expansion="tail"):
    """Speedup over the dense baseline per (token count, N:M) on another
    workload, with the compact weights expanded as in the main line: ABBA
    rounds with an event after every GEMM; reported beside the main line,
    never folded into its value."""
    work, preps = prepare(cfg, torch)
    if expansion == "tail":
        carry_expansions(preps)
    sp = [p.run_sparse for p in preps]
    dn = [p.run_dense for p in preps]
    abba(torch, sp, dn, 1, per_call=True)  # warm-up
    ta, tb = abba(torch, sp, dn, rounds, per_call=True)
    out = per_key_speedups(preps, ta.mean(axis=0), tb.mean(axis=0), lambda p: f"m={p.g.m} {pattern_name(p.g)}")
    del preps
    torch.cuda.empty_cache()
    return {"workload": work.name, "outputs": "int32", "order": "ABBA, event after every GEMM",
            "compact_weight_expansion": expansion, "per_batch_pattern": out}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=4,
                    help="0..4 (default 4: the 96 linears of ViT-L/16-384 at batch 32, layer-wise N:M)")
    ap.add_argument("--rounds", type=int, default=8, help="ABBA rounds of the speedup and control measurements")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the DeiT-Base per-batch speedups reported beside the main line")
    ap.add_argument("--no-mfma-ceiling", action="store_true",
                    help="skip the measured matrix-instruction rate reported beside the main line")
    ap.add_argument("--no-store-only", action="store_true",
                    help="skip the output-stream-only launches of the dominant kernel (keeps profiler traces to the "
                         "real launches)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after timing, run one plain device copy of MIB MiB (profiler counter calibration)")
    ap.add_argument("--expansion", choices=("tail", "call", "ahead"), default="tail",
                    help="where a plan that expands a compact weight once per call gets that expansion: 'tail' "
                         "(default) the previous GEMM's launch carries it (nm_spmm_out_expand) and the GEMM runs on "
                         "the expanded weight; 'call' inside the sparse call (nm_spmm's own expansion launch); "
                         "'ahead' nm_expand on a second stream with an event wait (measured slower on ViT-L: the "
                         "cross-stream waits cost more than the expansion latency they hide)")
    ap.add_argument("--traffic", type=str, default=None,
                    help="JSON record of measured HBM bytes per launch of the dominant kernel "
                         "(default: profiles/traffic_<workload>.json, used only if it matches this kernel source)")
    args = ap.parse_args()

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

    t0 = time.perf_counter()
    if args.expansion == "ahead":
        Prepared.side_stream = torch.cuda.Stream()   # default priority
    work, preps = prepare(args.config, torch)
    if args.expansion == "tail":
        carry_expansions(preps)
    out_i32, out_f16 = work.out_int32, work.out_f16
    log(f"workload {work.name}: {len(preps)} GEMMs, outputs {'int32' if out_i32 else ''}"
        f"{'+fp16' if out_f16 else ''}; inputs generated, packed and uploaded in {time.perf_counter() - t0:.1f} s")
    ops = np.array([p.g.dense_eq_ops for p in preps], np.float64)
    sp_calls = [p.run_sparse for p in preps]
    dn_calls = [p.run_dense for p in preps]

    # warm-up: untimed steps of both legs
    for _ in range(max(1, args.warmup)):
        for c in sp_calls + dn_calls:
            c()
    torch.cuda.synchronize()

    # the timed region: exactly K steps of the hot path
    ms_per_step, step_ev = timed_steps(preps, args.steps, torch)
    value = ops.sum() / (ms_per_step * 1e-3) / 1e12
    log(f"timed: {args.steps} steps, {ms_per_step:.4f} ms per step (events {step_ev.mean():.4f} ms), "
        f"{value:.1f} dense-equivalent TOPS")

    # speedup over the dense baseline (ABBA), and the A/A control
    rounds = max(2, args.rounds)
    ta, tb = abba(torch, sp_calls, dn_calls, rounds)
    speed = ratio_stats(ta, tb)
    ca, cb = abba(torch, dn_calls, dn_calls, rounds)
    control = ratio_stats(ca, cb)
    log(f"sparse leg {ta.mean():.4f} ms, dense leg {tb.mean():.4f} ms: speedup {speed['ratio']:.4f} "
        f"(rounds {speed['round_min']:.4f}..{speed['round_max']:.4f}); dense vs dense control "
        f"{control['ratio']:.4f} ({control['round_min']:.4f}..{control['round_max']:.4f})")

    # per GEMM (event after every GEMM), per pattern and per kernel
    pa, pb = abba(torch, sp_calls, dn_calls, max(2, rounds // 2), per_call=True)
    ts, td = pa.mean(axis=0), pb.mean(axis=0)
    per_pattern = per_key_speedups(preps, ts, td, lambda p: pattern_name(p.g))

    # dominant kernel: the sparse-leg kernel instantiation and GEMM shape with
    # the most time per step (one shape, so that a profiler's per-launch
    # average of that kernel and grid is the same quantity)
    kern = {}
    for i, p in enumerate(preps):
        k = kern.setdefault((p.kernel_name(p.splan), p.g.m, p.g.k, p.g.n), {"ms": 0.0, "idx": []})
        k["ms"] += ts[i]
        k["idx"].append(i)
    dom_key = max(kern, key=lambda k: kern[k]["ms"])
    dom_name = dom_key[0]
    dom_idx = kern[dom_key]["idx"]
    launches = len(dom_idx)
    # the kernel's own launch time: calls that also expand a compact weight
    # first (a second kernel inside the same call) are left out of the
    # average when calls without it exist
    plain = [i for i in dom_idx if not preps[i].expands_in_call()] or dom_idx
    avg_ms = float(np.mean([ts[i] for i in plain]))
    dom_bytes = sum(algorithmic_bytes(preps[i].g, out_i32, out_f16, sparse=preps[i].sparse_kernel) for i in dom_idx)
    dom_ops = sum(preps[i].g.dense_eq_ops for i in dom_idx)
    achieved = dom_bytes / launches / (avg_ms * 1e-3) / 1e9
    peak_ops = PEAK_SPARSE_TOPS if preps[dom_idx[0]].splan.kind in SP42_KINDS else PEAK_INT8_TOPS
    # which roofline binds: algorithmic bytes at the HBM peak against dense-equivalent ops at the matrix-core peak
    mfma_bound = dom_ops / (peak_ops * 1e12) > dom_bytes / (PEAK_HBM_GBS * 1e9)
    store_ms = None if args.no_store_only else store_only_time(preps, dom_idx, torch)
    traffic = None
    tpath = args.traffic or default_traffic_path(work.name)
    if os.path.exists(tpath):
        with open(tpath) as f:
            tr = json.load(f)
        # counters taken on another kernel (or an older build of it) do not count
        if (tr.get("kernel") == dom_name and tr.get("workload") == work.name
                and tr.get("grid") == int(preps[dom_idx[0]].splan.grid)
                and tr.get("kernel_source_sha256") == kernel_source_sha256()):
            traffic = tr.get("bytes_per_launch")
    if mfma_bound:
        achieved_ops = dom_ops / launches / (avg_ms * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved_ops, 1), "peak": peak_ops, "unit": "TOPS",
                    "frac": round(achieved_ops / peak_ops, 4)}
    else:
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roofline.update({
        "traffic": traffic,
        "kernel": dom_name,
        "gemm": {"m": dom_key[1], "k": dom_key[2], "n": dom_key[3],
                 "grid": int(preps[dom_idx[0]].splan.grid),
                 "patterns": sorted({pattern_name(preps[i].g) for i in dom_idx})},
        "launches_per_step": launches,
        "avg_launch_us": round(avg_ms * 1e3, 2),
        "avg_over_launches": len(plain),
        "algorithmic_bytes_per_launch": int(dom_bytes / launches),
        "algorithmic_ops_per_launch": int(dom_ops / launches),
        "hbm_gbs": round(achieved, 1),
        "share_of_step": round(float(kern[dom_key]["ms"] / ts.sum()), 3),
    })
    if store_ms is not None:
        # the same launches with the reduction skipped: the ceiling this
        # kernel's own output stream sets (context beside the HBM peak)
        roofline["output_stream_only_us"] = round(store_ms * 1e3, 2)
        roofline["frac_of_output_stream_only"] = round(store_ms / avg_ms, 3)

    log(f"\n{'gemm':<22}{'m':>7}{'k':>6}{'n':>6}  {'sparse kernel':<30}{'sparse us':>10}{'dense us':>10}"
        f"{'TOPS':>8}{'dTOPS':>8}{'spd':>7}{'GB/s':>8}")
    for i, p in enumerate(preps):
        g = p.g
        b = algorithmic_bytes(g, out_i32, out_f16, sparse=p.sparse_kernel)
        log(f"{g.name:<22}{g.m:>7}{g.k:>6}{g.n:>6}  {p.kernel_name(p.splan) + '/s' + str(p.splan.split_k):<30}"
            f"{ts[i] * 1e3:>10.1f}{td[i] * 1e3:>10.1f}{ops[i] / ts[i] / 1e9:>8.0f}{ops[i] / td[i] / 1e9:>8.0f}"
            f"{td[i] / ts[i]:>7.2f}{b / ts[i] / 1e6:>8.0f}")
    log(f"dominant kernel {dom_name}: {achieved:.0f} GB/s ({achieved / PEAK_HBM_GBS * 100:.1f}% of HBM peak), "
        f"{dom_ops / launches / (avg_ms * 1e-3) / 1e12:.0f} TOPS")

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
        "speedup_vs_dense": speed["ratio"],
        "speedup_rounds": speed,
        "control_dense_vs_dense": control,
        "sparse_leg_ms": round(float(ta.mean()), 4),
        "dense_leg_ms": round(float(tb.mean()), 4),
        "dense_tops": round(float(ops.sum() / (tb.mean() * 1e-3) / 1e12), 2),
        "step_event_ms": round(float(step_ev.mean()), 4),
        "frac_of_int8_peak": round(float(value / PEAK_INT8_TOPS), 4),
        "per_pattern": per_pattern,
        "cache_state": cache_state(preps),
        "compact_weight_expansion": {
            "tail": "carried by the previous GEMM's launch (nm_spmm_out_expand), for plans with expand = 1",
            "call": "in the sparse call",
            "ahead": "nm_expand on a second stream ahead of the GEMM, for plans with expand = 1"}[args.expansion],
        "roofline": roofline,
    }
    if not args.no_mfma_ceiling:
        line["mfma_measured"] = mfma_ceiling(torch)
        log(json.dumps(line["mfma_measured"]))
    if args.copy_calibration:
        # a plain elementwise pass that reads and writes exactly MIB MiB each
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        line["copy_calibration_bytes"] = 4 * n
        del src, dst
    if not args.no_cpu_baseline:
        cb, mism = cpu_baseline(preps, args.cpu_budget, check=True)
        line["cpu_baseline"] = cb
        line["parity_sampled_rows_mismatches"] = mism
        log(f"cpu oracle: {cb['value'] * 1e3:.2f} GOPS on {cb['cores']} threads; "
            f"GPU vs oracle on those rows: {mism} mismatches")
    else:
        line["cpu_baseline"] = None
    if not args.no_secondary and args.config != 2:
        del preps, sp_calls, dn_calls
        torch.cuda.empty_cache()
        line["deit_base_speedups"] = secondary_workload(2, max(2, rounds // 2), torch, args.expansion)
        log(json.dumps(line["deit_base_speedups"]))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
