"""Parity of the library's predictor and search (C ABI, include/nmsearch.h)
with the oracle (host code: CPU only).

* nm_nnls against the support-enumeration oracle on small problems (tolerance
  from the conditioning: backward-stable least squares on these well-conditioned
  random matrices agree to ~1e-13; 1e-9 relative leaves room), and against the
  optimality (KKT) conditions at the ViT-L calibration size (97 unknowns, over-
  and under-determined);
* nm_latency_fit / nm_latency_predict against the oracle's Eq. 1;
* nm_search against the oracle's Algorithm 1, configuration for configuration:
  both use the same counter-based generator and the same fitness function, so
  their results are identical.
"""
import math

import numpy as np
import pytest

from oracle import latency as orl
from oracle import search as ors
from paper_2607_12505_amd import nmsearch, nmspmm


def kkt_ok(A, y, x, tol=1e-9):
    w = A.T @ (y - A @ x)
    scale = np.abs(A).sum(axis=0).max() * max(1.0, np.abs(y).max())
    pos = x > 0
    return (x >= 0).all() and (np.abs(w[pos]) <= tol * scale).all() and (w[~pos] <= tol * scale).all()


@pytest.mark.parametrize("seed", range(16))
def test_nnls_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    rows, cols = int(rng.integers(4, 24)), int(rng.integers(1, 10))
    A = rng.standard_normal((rows, cols))
    if seed % 3 == 0:
        A = np.abs(A) * 10            # positive tables, like latencies
    y = rng.standard_normal(rows) * 5 + (A.sum(axis=1) if seed % 2 else 0)
    x, r = nmsearch.nnls(A, y)
    xo, ro = orl.nnls(A, y)
    assert r == pytest.approx(ro, rel=1e-9, abs=1e-12)
    if rows >= cols:
        assert np.allclose(x, xo, rtol=1e-9, atol=1e-11)
    assert kkt_ok(A, y, x)


@pytest.mark.parametrize("rows", [24, 150])
def test_nnls_kkt_at_calibration_size(rows):
    rng = np.random.default_rng(rows)
    t = rng.uniform(20, 120, (rows, 96))
    A = np.hstack([t, np.ones((rows, 1))])
    gamma = rng.uniform(0.5, 1.2, 96)
    gamma[rng.integers(0, 96, 10)] = 0.0
    y = A[:, :96] @ gamma + 40.0 + rng.normal(0, 5.0, rows)
    x, r = nmsearch.nnls(A, y)
    assert kkt_ok(A, y, x)
    assert r == pytest.approx(np.linalg.norm(A @ x - y), rel=1e-9, abs=1e-12 * np.linalg.norm(y))


def test_nnls_errors_and_degenerate_columns():
    with pytest.raises(nmspmm.NmError) as e:
        nmsearch.nnls(np.array([[1.0, np.nan]]), np.array([1.0]))
    assert e.value.status == nmspmm.NM_ERR_ARG
    # duplicated column: the fit is still optimal, one copy stays at zero or they share
    A = np.array([[1.0, 1.0, 0.0], [2.0, 2.0, 1.0], [3.0, 3.0, 1.0]])
    y = np.array([1.0, 3.0, 4.0])
    x, r = nmsearch.nnls(A, y)
    _, ro = orl.nnls(A, y)
    assert r == pytest.approx(ro, abs=1e-10) and (x >= 0).all()
    # zero matrix: x = 0
    x, r = nmsearch.nnls(np.zeros((3, 2)), np.array([1.0, 2.0, 2.0]))
    assert (x == 0).all() and r == pytest.approx(3.0)


def test_latency_fit_and_predict_match_oracle():
    rng = np.random.default_rng(8)
    L, K = 6, 14
    t_rows = rng.uniform(10, 80, (K, L))
    T = t_rows @ rng.uniform(0.7, 1.3, L) + 12.0 + rng.normal(0, 1.0, K)
    g, b = nmsearch.latency_fit(t_rows, T)
    go, bo = orl.fit(t_rows, T)
    assert np.allclose(g, go, rtol=1e-9, atol=1e-10) and b == pytest.approx(bo, rel=1e-9, abs=1e-10)
    for row in t_rows:
        assert nmsearch.latency_predict(row, g, b) == orl.predict(row, g, b)   # same order of the sum


def vit_large_problem(seed, L=96):
    """A ViT-L-shaped table: 4 GEMM shapes repeated over 24 blocks, latency
    growing with N, per-layer gamma near 1; concave separable accuracy."""
    rng = np.random.default_rng(seed)
    shape_base = [60.0, 22.0, 80.0, 75.0]
    lut = []
    for l in range(L):
        base = shape_base[l % 4]
        lut.append([float(base * (0.45 + 0.55 * n / 8) * rng.uniform(0.97, 1.03)) for n in range(1, 9)])
    gamma = rng.uniform(0.85, 1.1, L).tolist()
    b = float(rng.uniform(5, 30))
    sens = rng.uniform(0.05, 1.0, L)
    acc = lambda y: float(sum(sens[l] * math.log(y[l] / 8.0) for l in range(L)))
    lo = sum(g * t[0] for g, t in zip(gamma, lut)) + b
    hi = sum(g * t[7] for g, t in zip(gamma, lut)) + b
    return lut, gamma, b, lo, hi, acc


@pytest.mark.parametrize("seed,frac", [(0, 0.5), (1, 0.3), (2, 0.7), (3, 0.05)])
def test_search_matches_oracle(seed, frac):
    lut, gamma, b, lo, hi, acc = vit_large_problem(seed)
    target = lo + frac * (hi - lo)
    got = nmsearch.search(lut, gamma, b, target, acc, generations=5, offspring=4, overshoot=4, seed=seed + 10)
    want = ors.search(lut, gamma, b, target, acc, 5, 4, 4, seed + 10)
    assert got[0] == want[0]
    assert got[1] == want[1]
    assert got[2] == want[2]


def test_search_edge_cases():
    lut, gamma, b, lo, hi, acc = vit_large_problem(5, L=8)
    # budget below the sparsest uniform configuration
    with pytest.raises(nmspmm.NmError) as e:
        nmsearch.search(lut, gamma, b, lo * 0.9, acc, 2, 2, 1, seed=1)
    assert e.value.status == nmspmm.NM_ERR_SHAPE
    # generous budget: all dense; zero generations: the initial configuration
    x, f, trace = nmsearch.search(lut, gamma, b, hi * 2, acc, 0, 2, 1, seed=1)
    assert x == [8] * 8 and trace == [f]
    # bad parameters
    with pytest.raises(nmspmm.NmError):
        nmsearch.search(lut, gamma, b, hi, acc, 1, 0, 1, seed=1)
    # an exception inside the fitness is re-raised after the call
    def boom(y):
        raise ValueError("fitness failed")
    with pytest.raises(ValueError):
        nmsearch.search(lut, gamma, b, hi, boom, 1, 1, 1, seed=1)
