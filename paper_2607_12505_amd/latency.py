"""Operator latency table and whole-chain timing for the layer-wise search
(paper Sec. 5.1).

The table (LUT) maps (GEMM shape, N:M pattern, outputs) to the mean latency
of the library's GEMM over repeated runs; a configuration's end-to-end
latency is then predicted by Eq. 1 (nm_latency_fit / nm_latency_predict in
the library).  Full-model measurements time a whole chain of linears
back-to-back on one stream.  Every GEMM runs in libnmspmm; PyTorch provides
device memory, the stream and HIP events.
"""
from __future__ import annotations

import ctypes
import json
import time
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import nmspmm
from . import workloads as wl

FAMILY_N8 = tuple((n, 8) for n in range(1, 9))   # the search space: N:8, N = 8 is dense

Shape = Tuple[int, int, int]          # (m, k, n)
Pattern = Tuple[int, int]             # (N, M)


class GemmCall:
    """One GEMM (shape, pattern) with resident inputs and prepared C arguments.
    Dense patterns (N == M) run the dense GEMM."""

    def __init__(self, torch, shape: Shape, pattern: Pattern, X, Y, Yh, scale, seed: int, out_mode: int):
        m, k, n = shape
        N, M = pattern
        self.shape, self.pattern = shape, pattern
        W, _ = wl.gen_w(n, k, N, M, np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, m, k, n, N,
                                                                                                  M]))))
        L = nmspmm.lib()
        ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        y = Y if out_mode & nmspmm.NM_OUT_I32 else None
        yh = Yh if out_mode & nmspmm.NM_OUT_F16 else None
        self.dense = N == M
        if self.dense:
            self.W = torch.from_numpy(W).cuda()
            self.plan = nmspmm.dense_plan(m, n, k, out_mode)
        else:
            packed = nmspmm.compress(W, N, M)
            self.dw = nmspmm.DeviceWeight.from_packed(packed)
            self.plan = nmspmm.spmm_plan(packed.desc, m, out_mode)
        need = nmspmm.workspace_size(self.plan, m, n)
        self.ws = torch.zeros(max(need, 16), dtype=torch.uint8, device="cuda")
        if self.dense:
            self.fn = L.nm_gemm_i8_dense_ex
            self.args = (ptr(X), m, ptr(self.W), n, k, ptr(y), ptr(scale), ptr(yh), ptr(self.ws), self.ws.numel(),
                         stream, ctypes.byref(self.plan))
        else:
            self.fn = L.nm_spmm_ex
            self.args = (ptr(X), m, ptr(self.dw.vals), ptr(self.dw.meta), ctypes.byref(self.dw.desc), ptr(y),
                         ptr(scale), ptr(yh), ptr(self.ws), self.ws.numel(), stream, ctypes.byref(self.plan))

    def __call__(self):
        st = self.fn(*self.args)
        if st:
            raise nmspmm.NmError(st, f"GEMM {self.shape} {self.pattern}")


def time_launches(torch, fn, reps: int, windows: int = 3) -> float:
    """Microseconds per call over `reps` back-to-back calls, bracketed by HIP
    events on the current stream after a device sleep meant to outlast the
    host's queueing of every call, so that the GPU runs them back to back.
    A window in which the host took longer to queue the calls than the sleep
    lasted (a host stall reached the GPU timeline) does not count; of the
    `windows` windows the fastest valid one is returned (the fastest of all
    if none is valid)."""
    fn()
    torch.cuda.synchronize()
    sleep_s = 150e-6 * reps
    valid, every = [], []
    for _ in range(windows):
        # the sleep is given in cycles at the top clock, so it lasts at least sleep_s
        torch.cuda._sleep(int(2.4e9 * sleep_s))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        h0 = time.perf_counter()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        host = time.perf_counter() - h0
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e3 / reps
        every.append(t)
        if host < sleep_s:
            valid.append(t)
    return min(valid) if valid else min(every)


def time_cold(torch, fn, reps: int, flush) -> float:
    """Mean microseconds of single calls that each start with cold caches: a
    write over `flush` (a buffer larger than L2 and the last-level cache)
    precedes every call, outside its event pair."""
    fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for e0, e1 in ev:
        flush.fill_(1)
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev])) * 1e3


class ChainBench:
    """The GEMMs of a chain of linears (one shape per position) under every
    pattern of a set, sharing one input buffer per (m, k) and one output
    buffer per (m, n)."""

    def __init__(self, torch, layer_shapes: Sequence[Shape], patterns: Sequence[Pattern],
                 out_mode: int = nmspmm.NM_OUT_I32, seed: int = 0):
        self.torch = torch
        self.layer_shapes = list(layer_shapes)
        self.patterns = list(patterns)
        self.out_mode = out_mode
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 77])))
        xs: Dict[Tuple[int, int], object] = {}
        ys: Dict[Tuple[int, int], tuple] = {}
        self.calls: Dict[Tuple[Shape, Pattern], GemmCall] = {}
        for shape in dict.fromkeys(self.layer_shapes):
            m, k, n = shape
            if (m, k) not in xs:
                xs[(m, k)] = torch.from_numpy(wl.gen_x(m, k, rng)).cuda()
            if (m, n) not in ys:
                Y = torch.empty((m, n), dtype=torch.int32, device="cuda") if out_mode & nmspmm.NM_OUT_I32 else None
                Yh = torch.empty((m, n), dtype=torch.int16, device="cuda") if out_mode & nmspmm.NM_OUT_F16 else None
                sc = torch.full((n,), 1e-4, dtype=torch.float32, device="cuda")
                ys[(m, n)] = (Y, Yh, sc)
            Y, Yh, sc = ys[(m, n)]
            for pat in self.patterns:
                self.calls[(shape, pat)] = GemmCall(torch, shape, pat, xs[(m, k)], Y, Yh, sc, seed, out_mode)
        self._keep = (xs, ys)
        torch.cuda.synchronize()

    def lut(self, reps: int = 20, cold: bool = True) -> Tuple[Dict[Tuple[Shape, Pattern], float], float]:
        """Mean latency of every (shape, pattern) over `reps` runs; also the
        wall seconds it took.  cold: each run starts with flushed caches, as a
        linear inside a network does (its input was written long before);
        otherwise back-to-back repeats on the same, cache-resident, input."""
        t0 = time.perf_counter()
        if cold:
            flush = self.torch.empty(512 << 20, dtype=self.torch.uint8, device="cuda")
            table = {key: time_cold(self.torch, call, reps, flush) for key, call in self.calls.items()}
            del flush
        else:
            table = {key: time_launches(self.torch, call, reps) for key, call in self.calls.items()}
        return table, time.perf_counter() - t0

    def layer_times(self, table, assignment: Sequence[Pattern]) -> List[float]:
        """t_l(s_l) of every layer of a configuration."""
        return [table[(shape, pat)] for shape, pat in zip(self.layer_shapes, assignment)]

    def measure(self, assignment: Sequence[Pattern], reps: int = 3) -> float:
        """Mean end-to-end microseconds of the whole chain under a configuration."""
        calls = [self.calls[(shape, pat)] for shape, pat in zip(self.layer_shapes, assignment)]

        def chain():
            for c in calls:
                c()

        torch = self.torch
        chain()
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 25e-6 * len(calls)))
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record()
        for r in range(reps):
            chain()
            ev[r + 1].record()
        torch.cuda.synchronize()
        return float(np.mean([ev[r].elapsed_time(ev[r + 1]) * 1e3 for r in range(reps)]))


def vit_large_layer_shapes(batch: int = 32) -> List[Shape]:
    """The 96 linears of ViT-L/16 at 384 px: (m, k, n) per position."""
    m, C, H = batch * 577, 1024, 4096
    per_block = [(m, C, 3 * C), (m, C, C), (m, C, H), (m, H, C)]
    return per_block * 24


def random_assignments(count: int, layers: int, patterns: Sequence[Pattern], seed: int) -> List[List[Pattern]]:
    """Configurations with one uniform pattern draw per layer."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 4242])))
    return [[patterns[int(i)] for i in rng.integers(0, len(patterns), layers)] for _ in range(count)]


# ---------------------------------------------------------------------------
# Persistence: the table is built once offline and reused by every search, so
# it is kept as JSON together with the calibration of Eq. 1 (gamma, b) and a
# free-form record of where it was measured.

LUT_FORMAT = "nmspmm-lut/1"


def save_lut(path: str, table: Dict[Tuple[Shape, Pattern], float], gamma: Optional[Sequence[float]] = None,
             b: Optional[float] = None, info: Optional[dict] = None) -> None:
    """Writes the table (and, if given, the calibrated gamma and b) as JSON."""
    entries = [{"m": m, "k": k, "n": n, "N": N, "M": M, "us": float(t)}
               for ((m, k, n), (N, M)), t in sorted(table.items())]
    doc = {"format": LUT_FORMAT, "entries": entries, "info": info or {}}
    if gamma is not None:
        doc["gamma"] = [float(g) for g in gamma]
        doc["b"] = float(b if b is not None else 0.0)
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)


def load_lut(path: str) -> Tuple[Dict[Tuple[Shape, Pattern], float], Optional[List[float]], Optional[float], dict]:
    """Reads a file written by save_lut: (table, gamma or None, b or None, info).
    Raises ValueError on another format, a duplicate key or a latency that is
    not a finite non-negative number."""
    with open(path) as f:
        doc = json.load(f)
    if doc.get("format") != LUT_FORMAT:
        raise ValueError(f"{path}: not a {LUT_FORMAT} file")
    table: Dict[Tuple[Shape, Pattern], float] = {}
    for e in doc["entries"]:
        key = ((int(e["m"]), int(e["k"]), int(e["n"])), (int(e["N"]), int(e["M"])))
        t = float(e["us"])
        if key in table:
            raise ValueError(f"{path}: duplicate entry {key}")
        if not np.isfinite(t) or t < 0:
            raise ValueError(f"{path}: bad latency {t} for {key}")
        table[key] = t
    gamma = [float(g) for g in doc["gamma"]] if "gamma" in doc else None
    b = float(doc["b"]) if "b" in doc else None
    return table, gamma, b, doc.get("info", {})
