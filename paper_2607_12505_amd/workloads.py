"""Seeded synthetic inputs for the N:M sparse INT8 GEMM, and the benchmark shapes.

This module only draws inputs.  It holds none of the GEMM's arithmetic and is
shared by the HIP path's tests/benchmark and by the oracle's tests, which is
why it sits in a module of its own.

Recipe (the paper evaluates on ViT/DeiT/Swin linears, Sec. 6; no dataset or
trained weight is needed, only the GEMM shapes):

* X: integers uniform on [-127, 127] (int8 activations).
* W: float64 N(0, 0.02) -> keep the N largest magnitudes in every aligned
  window of M along k (ties go to the lower index) -> symmetric per-row int8
  quantisation s_w = max|w| / 127, q = clip(round_half_even(w / s_w), -127, 127)
  (an all-zero row gets s_w = 1).  A kept weight that rounds to zero stays
  zero, so windows hold *at most* N nonzeros.
* scale[j] = s_w[j] / 127 as float32: the per-output-channel dequantisation
  factor for activations quantised with s_x = 1/127.
* Every draw comes from PCG64 seeded by SeedSequence([cfg, layer, linear, pattern, role]).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

ROLE_X, ROLE_W = 0, 1


def rng_for(cfg: int, layer: int, linear: int, pattern: int, role: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg, layer, linear, pattern, role])))


def gen_x(m: int, k: int, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(-127, 128, size=(m, k), dtype=np.int8)


def gen_w(n: int, k: int, N: int, M: int, rng: np.random.Generator) -> Tuple[np.ndarray, np.ndarray]:
    """Returns (W int8 [n, k] with at most N nonzeros per aligned M-window, scale float32 [n])."""
    if k % M != 0:
        raise ValueError("k must be a multiple of M")
    w = rng.normal(0.0, 0.02, size=(n, k))
    if N < M:
        groups = w.reshape(n, k // M, M)
        # stable sort of -|w| keeps the lower index first among equal magnitudes
        order = np.argsort(-np.abs(groups), axis=2, kind="stable")
        keep = np.zeros_like(groups, dtype=bool)
        np.put_along_axis(keep, order[:, :, :N], True, axis=2)
        w = np.where(keep, groups, 0.0).reshape(n, k)
    amax = np.abs(w).max(axis=1)
    s_w = np.where(amax > 0, amax / 127.0, 1.0)
    q = np.clip(np.rint(w / s_w[:, None]), -127, 127).astype(np.int8)
    scale = (s_w / 127.0).astype(np.float32)
    return q, scale


# ---------------------------------------------------------------------------
# Benchmark shapes: ViT-family linears (m tokens, k in_features, n out_features)

@dataclasses.dataclass(frozen=True)
class Gemm:
    name: str
    m: int
    k: int
    n: int
    N: int  # nonzeros per window (N == M means dense)
    M: int
    layer: int = 0
    linear: int = 0

    @property
    def dense_eq_ops(self) -> int:
        return 2 * self.m * self.n * self.k


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    gemms: Tuple[Gemm, ...]
    out_int32: bool = True
    out_f16: bool = False
    chain: bool = False  # one back-to-back sequence (a whole network's linears)


PATTERN_IDS = {(1, 4): 0, (2, 4): 1, (1, 8): 2, (2, 8): 3, (4, 8): 4, (4, 4): 5, (8, 8): 5}


def _vit_block(prefix: str, m: int, C: int, hidden: int, N: int, M: int, layer: int = 0) -> List[Gemm]:
    return [
        Gemm(f"{prefix}qkv", m, C, 3 * C, N, M, layer, 0),
        Gemm(f"{prefix}proj", m, C, C, N, M, layer, 1),
        Gemm(f"{prefix}fc1", m, C, hidden, N, M, layer, 2),
        Gemm(f"{prefix}fc2", m, hidden, C, N, M, layer, 3),
    ]


def workload(cfg: int) -> Workload:
    if cfg == 0:
        return Workload(0, "deit_tiny_fc1_b1", (Gemm("fc1", 197, 192, 768, 2, 4, 0, 2),))
    if cfg == 1:
        g = []
        for (N, M) in ((1, 4), (2, 4), (2, 8), (4, 8)):
            g += _vit_block(f"{N}:{M} ", 64 * 197, 384, 1536, N, M)
        return Workload(1, "deit_small_b64", tuple(g), out_int32=True, out_f16=True)
    if cfg == 2:
        g = []
        for b in (1, 8, 128):
            for (N, M) in ((1, 4), (2, 4), (1, 8), (2, 8)):
                g += _vit_block(f"b{b} {N}:{M} ", b * 197, 768, 3072, N, M)
        return Workload(2, "deit_base_b1_b8_b128", tuple(g))
    if cfg == 3:
        g = []
        for (C, tok) in ((128, 3136), (256, 784), (512, 196), (1024, 49)):
            for (N, M) in ((2, 4), (2, 8)):
                g += _vit_block(f"C{C} {N}:{M} ", 32 * tok, C, 4 * C, N, M)
        return Workload(3, "swin_b_b32", tuple(g))
    if cfg == 4:
        return Workload(4, "vit_large_384_b32_chain", tuple(vit_large_chain()), chain=True)
    raise ValueError(f"no workload {cfg}")


VIT_L_CHOICES = ((8, 8), (4, 8), (2, 4), (2, 8), (1, 4))


def vit_large_assignment(seed: int = 4) -> List[Tuple[int, int]]:
    """Layer-wise N:M draw for the 24x4 ViT-L/16 linears: one uniform draw per linear."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 9999])))
    picks = rng.integers(0, len(VIT_L_CHOICES), size=96)
    return [VIT_L_CHOICES[int(p)] for p in picks]


def vit_large_chain(seed: int = 4) -> List[Gemm]:
    assign = vit_large_assignment(seed)
    m, C, H = 32 * 577, 1024, 4096
    shapes = (("qkv", C, 3 * C), ("proj", C, C), ("fc1", C, H), ("fc2", H, C))
    g = []
    for layer in range(24):
        for lin, (nm, k, n) in enumerate(shapes):
            N, M = assign[layer * 4 + lin]
            g.append(Gemm(f"L{layer} {nm} {N}:{M}", m, k, n, N, M, layer, lin))
    return g


def inputs_for(cfg: int, gm: Gemm, x_cache: Optional[dict] = None):
    """(X, W, scale) for one GEMM of a workload, all deterministic in (cfg, gemm)."""
    pid = PATTERN_IDS.get((gm.N, gm.M), 7)
    key = (gm.m, gm.k, gm.layer, gm.linear)
    if x_cache is not None and key in x_cache:
        X = x_cache[key]
    else:
        X = gen_x(gm.m, gm.k, rng_for(cfg, gm.layer, gm.linear, 0, ROLE_X))
        if x_cache is not None:
            x_cache[key] = X
    W, scale = gen_w(gm.n, gm.k, gm.N, gm.M, rng_for(cfg, gm.layer, gm.linear, pid, ROLE_W))
    return X, W, scale


def random_nm(n: int, k: int, N: int, M: int, rng: np.random.Generator, full: bool = False,
              extremes: bool = True) -> np.ndarray:
    """Random int8 matrix with 0..N nonzeros (exactly N if full) per aligned window,
    values drawn from the whole int8 range (edge values -128/127 included)."""
    G = k // M
    cnt = np.full((n, G), N) if full else rng.integers(0, N + 1, size=(n, G))
    # a uniformly random subset of cnt positions per window: ranks of random keys
    rank = np.argsort(np.argsort(rng.random((n, G, M)), axis=2), axis=2)
    lo = -128 if extremes else -127
    v = rng.integers(lo, 128, size=(n, G, M))
    v[v == 0] = 1
    return np.where(rank < cnt[..., None], v, 0).astype(np.int8).reshape(n, k)
