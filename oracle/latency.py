"""Oracle of the LUT latency predictor (paper Sec. 5.1, Eq. 1) -- test
infrastructure only (tests, smoke check and benchmark baseline use it; the
product library never does).

* ``predict``: T_pred = sum_l gamma_l * t_l(s_l) + b, a plain loop in the
  order of the sum.
* ``nnls``: the non-negative least-squares calibration of (gamma, b), solved
  by its definition: the minimiser of ||A x - y|| over x >= 0 is, on its
  support S, the unconstrained least-squares solution on the columns in S.  So
  enumerating every subset S, solving least squares on S, keeping the
  solutions that are non-negative and taking the smallest residual gives the
  optimum.  2^cols subsets: tiny problems only.
* ``fit``: Eq. 1's calibration -- the design matrix holds each measured
  configuration's LUT latencies per layer plus a column of ones for b.
"""
import itertools

import numpy as np


def predict(t, gamma, b):
    """T_pred of one configuration: t[l] is the LUT latency of layer l under
    its sparsity setting."""
    total = 0.0
    for tl, gl in zip(t, gamma):
        total += gl * tl
    return total + b


def nnls(A, y):
    """Returns (x, residual norm) minimising ||A x - y||_2 subject to x >= 0,
    by enumeration of supports (cols <= 14)."""
    A = np.asarray(A, np.float64)
    y = np.asarray(y, np.float64)
    rows, cols = A.shape
    if cols > 14:
        raise ValueError("brute force is for tiny problems")
    best_x, best_r = np.zeros(cols), float(np.linalg.norm(y))
    for size in range(1, cols + 1):
        for S in itertools.combinations(range(cols), size):
            S = list(S)
            xs, *_ = np.linalg.lstsq(A[:, S], y, rcond=None)
            if (xs < 0).any():
                continue
            x = np.zeros(cols)
            x[S] = xs
            r = float(np.linalg.norm(A @ x - y))
            if r < best_r:
                best_x, best_r = x, r
    return best_x, best_r


def design_matrix(t_rows):
    """Rows [t_1(s_1), ..., t_L(s_L), 1] of the calibration configurations."""
    t_rows = np.asarray(t_rows, np.float64)
    return np.hstack([t_rows, np.ones((t_rows.shape[0], 1))])


def fit(t_rows, T):
    """(gamma, b) of Eq. 1 by NNLS on the measured latencies T."""
    x, _ = nnls(design_matrix(t_rows), T)
    return x[:-1], x[-1]
