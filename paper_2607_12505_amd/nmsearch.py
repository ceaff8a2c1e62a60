"""Thin ctypes binding of the predictor and search entry points (C ABI in
include/nmsearch.h, same library as the GEMMs).  Host arrays only; every step
runs in the library."""
from __future__ import annotations

import ctypes

import numpy as np

from . import nmspmm

EXPORTED = ("nm_nnls", "nm_latency_fit", "nm_latency_predict", "nm_search")

FITNESS_FN = ctypes.CFUNCTYPE(ctypes.c_double, ctypes.POINTER(ctypes.c_int32), ctypes.c_int, ctypes.c_void_p)


class NmSearchParams(ctypes.Structure):
    _fields_ = [("generations", ctypes.c_int32), ("offspring", ctypes.c_int32), ("overshoot", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("seed", ctypes.c_uint64)]


_sigs_done = False


def _lib():
    global _sigs_done
    L = nmspmm.lib()
    if not _sigs_done:
        dp, i32 = ctypes.POINTER(ctypes.c_double), ctypes.c_int
        L.nm_nnls.argtypes = [dp, i32, i32, dp, dp, dp]
        L.nm_latency_fit.argtypes = [dp, i32, i32, dp, dp, dp]
        L.nm_latency_predict.argtypes = [dp, i32, dp, ctypes.c_double, dp]
        L.nm_search.argtypes = [i32, dp, dp, ctypes.c_double, ctypes.c_double, FITNESS_FN, ctypes.c_void_p,
                                ctypes.POINTER(NmSearchParams), ctypes.POINTER(ctypes.c_int32), dp, dp]
        for f in (L.nm_nnls, L.nm_latency_fit, L.nm_latency_predict, L.nm_search):
            f.restype = i32
        _sigs_done = True
    return L


def _d(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _check(st, what):
    if st != nmspmm.NM_OK:
        raise nmspmm.NmError(st, what)


def nnls(A, y):
    """(x, ||A x - y||) with x >= 0 minimising the residual (nm_nnls)."""
    A, y = _d(A), _d(y)
    rows, cols = A.shape
    x = np.zeros(cols)
    r = ctypes.c_double()
    _check(_lib().nm_nnls(_p(A), rows, cols, _p(y), _p(x), ctypes.byref(r)), "nm_nnls")
    return x, r.value


def latency_fit(t_rows, T):
    """(gamma, b) of Eq. 1 from [configs x layers] table latencies and measured T (nm_latency_fit)."""
    t_rows, T = _d(t_rows), _d(T)
    K, L = t_rows.shape
    gamma = np.zeros(L)
    b = ctypes.c_double()
    _check(_lib().nm_latency_fit(_p(t_rows), K, L, _p(T), _p(gamma), ctypes.byref(b)), "nm_latency_fit")
    return gamma, b.value


def latency_predict(t, gamma, b):
    t, gamma = _d(t), _d(gamma)
    out = ctypes.c_double()
    _check(_lib().nm_latency_predict(_p(t), t.size, _p(gamma), float(b), ctypes.byref(out)), "nm_latency_predict")
    return out.value


def search(lut, gamma, b, target, accuracy, generations, offspring, overshoot, seed):
    """Algorithm 1 (nm_search).  lut [layers x 8] with lut[l][N-1] = t_l(N:8);
    accuracy(list of N per layer) -> float.  Returns (config, fitness, trace)."""
    lut, gamma = _d(lut), _d(gamma)
    L = lut.shape[0]
    errors = []

    def cb(ptr, n, _user):
        try:
            return float(accuracy([ptr[i] for i in range(n)]))
        except BaseException as e:  # noqa: BLE001 - reported after the call
            errors.append(e)
            return float("nan")

    fn = FITNESS_FN(cb)
    params = NmSearchParams(generations, offspring, overshoot, 0, seed & ((1 << 64) - 1))
    best = np.zeros(L, np.int32)
    fit = ctypes.c_double()
    trace = np.zeros(generations + 1)
    st = _lib().nm_search(L, _p(lut), _p(gamma), float(b), float(target), fn, None, ctypes.byref(params),
                          best.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), ctypes.byref(fit), _p(trace))
    if errors:
        raise errors[0]
    _check(st, "nm_search")
    return best.tolist(), fit.value, trace.tolist()
