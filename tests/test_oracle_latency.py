"""Pins of the latency-predictor oracle (Eq. 1 and its NNLS calibration)
against things other than itself: SciPy's NNLS (an independent active-set
implementation), the optimality (KKT) conditions, closed forms and exactly
representable configurations.  CPU only."""
import numpy as np
import pytest
import scipy.optimize

from oracle import latency as orl


def kkt_ok(A, y, x, tol=1e-8):
    """x >= 0; the gradient A^T (y - A x) is <= 0 where x = 0 and 0 where x > 0."""
    w = A.T @ (y - A @ x)
    scale = np.abs(A).sum() * max(1.0, np.abs(y).max())
    pos = x > 1e-12
    return (x >= 0).all() and (np.abs(w[pos]) <= tol * scale).all() and (w[~pos] <= tol * scale).all()


@pytest.mark.parametrize("seed", range(12))
def test_nnls_matches_scipy_and_kkt(seed):
    rng = np.random.default_rng(seed)
    rows, cols = int(rng.integers(3, 20)), int(rng.integers(1, 9))
    A = rng.standard_normal((rows, cols))
    y = rng.standard_normal(rows) * 3
    x, r = orl.nnls(A, y)
    xs, rs = scipy.optimize.nnls(A, y)
    assert r == pytest.approx(rs, rel=1e-9, abs=1e-12)
    if rows >= cols:          # full column rank (almost surely): the minimiser is unique
        assert np.allclose(x, xs, rtol=1e-8, atol=1e-10)
    assert kkt_ok(A, y, x)


def test_nnls_closed_forms():
    # one column: x = max(0, a.y / a.a)
    a = np.array([[1.0], [2.0], [2.0]])
    x, r = orl.nnls(a, np.array([1.0, 1.0, 4.0]))
    assert x[0] == pytest.approx(11.0 / 9.0)
    x, r = orl.nnls(a, np.array([-1.0, -1.0, -4.0]))
    assert x[0] == 0.0 and r == pytest.approx(np.sqrt(18.0))
    # an unconstrained solution that is already non-negative is the answer
    A = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    y = A @ np.array([2.0, 3.0])
    x, r = orl.nnls(A, y)
    assert np.allclose(x, [2.0, 3.0]) and r == pytest.approx(0.0, abs=1e-12)
    # a negative unconstrained coefficient is clamped and the rest refitted
    A = np.eye(3)
    x, r = orl.nnls(A, np.array([1.0, -2.0, 3.0]))
    assert np.allclose(x, [1.0, 0.0, 3.0]) and r == pytest.approx(2.0)


def test_predict_is_the_weighted_sum():
    t = [10.0, 20.0, 5.0]
    assert orl.predict(t, [1.0, 0.5, 2.0], 3.0) == 10.0 + 10.0 + 10.0 + 3.0
    assert orl.predict(t, [0.0, 0.0, 0.0], 0.0) == 0.0


def test_fit_recovers_an_exact_model():
    rng = np.random.default_rng(4)
    L, K = 5, 12
    t_rows = rng.uniform(10, 100, (K, L))
    gamma = np.array([1.0, 0.8, 1.2, 0.0, 0.5])
    b = 7.0
    T = np.array([orl.predict(r, gamma, b) for r in t_rows])
    g, bb = orl.fit(t_rows, T)
    assert np.allclose(g, gamma, atol=1e-9) and bb == pytest.approx(b, abs=1e-8)
    # an intercept the data pushes negative is clamped to zero
    T2 = t_rows.sum(axis=1) - 50.0
    g2, b2 = orl.fit(t_rows, T2)
    assert b2 == 0.0 and (g2 >= 0).all()
