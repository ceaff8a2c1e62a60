"""CPU oracle for the N:M sparse INT8 GEMM -- test infrastructure only.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It wraps ``oracle.c`` (plain C, exact integer arithmetic,
one rounding to binary16) through ctypes and shares nothing with the HIP
library.  Functions follow the paper's definitions:

* ``nm_check``            -- N:M validity of every aligned window (Sec. 2.1)
* ``pack_logical`` / ``unpack_logical`` -- B_pack as values plus in-window
  positions (Sec. 4.2), canonical slot order
* ``spmm_packed``         -- the product evaluated from the packed form (Sec. 4.2)
* ``matmul_i8``           -- the plain product Y = X W^T (its definition)
* ``dequant_f16`` / ``f64_to_f16`` -- per-channel dequantisation, one rounding
* ``quantize_f16`` / ``requant_i8`` / ``f16_to_f32`` -- int8 quantisation on
  either side of a linear in INT8 deployment (Sec. 6.3), decided in binary32
"""
import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, ERR_ARG, ERR_OVERFLOW, ERR_PATTERN = 0, 1, 2, 3

_i8p = ctypes.POINTER(ctypes.c_int8)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    src = os.path.join(_HERE, "oracle.c")
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    c_int = ctypes.c_int
    lib.orc_nm_check.argtypes = [_i8p, c_int, c_int, c_int, c_int, _ip, _ip]
    lib.orc_pack_logical.argtypes = [_i8p, c_int, c_int, c_int, c_int, _i8p, _u8p]
    lib.orc_unpack_logical.argtypes = [_i8p, _u8p, c_int, c_int, c_int, c_int, _i8p]
    lib.orc_matmul_i8.argtypes = [_i8p, _i8p, c_int, c_int, c_int, _i32p, c_int]
    lib.orc_matmul_i8_sampled.argtypes = [_i8p, _i8p, c_int, c_int, c_int, _i64p, _i64p,
                                          ctypes.c_int64, _i32p]
    lib.orc_spmm_packed.argtypes = [_i8p, c_int, _i8p, _u8p, c_int, c_int, c_int, c_int, _i32p, c_int]
    lib.orc_f64_to_f16.argtypes = [ctypes.c_double]
    lib.orc_f64_to_f16.restype = ctypes.c_uint16
    lib.orc_f64_to_f16_array.argtypes = [_f64p, ctypes.c_int64, _u16p]
    lib.orc_dequant_f16.argtypes = [_i32p, _f32p, c_int, c_int, _u16p]
    lib.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_f16_to_f32.restype = ctypes.c_float
    lib.orc_quantize_f16.argtypes = [_u16p, ctypes.c_int64, ctypes.c_float, _i8p]
    lib.orc_requant_i8.argtypes = [_i32p, _f32p, c_int, c_int, _i8p]
    for f in (lib.orc_nm_check, lib.orc_pack_logical, lib.orc_unpack_logical, lib.orc_matmul_i8,
              lib.orc_matmul_i8_sampled, lib.orc_spmm_packed, lib.orc_dequant_f16, lib.orc_quantize_f16,
              lib.orc_requant_i8):
        f.restype = c_int
    _lib = lib
    return lib


def _ptr(a, t):
    return a.ctypes.data_as(t)


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
    return a


class OracleError(RuntimeError):
    pass


def _check(rc, what):
    if rc != OK:
        raise OracleError(f"{what}: oracle status {rc}")


def nm_check(W, N, M):
    """Returns (ok, bad_row, bad_group) for the N:M rule along the last axis."""
    W = _c(W, np.int8)
    n, k = W.shape
    br, bg = ctypes.c_int(-1), ctypes.c_int(-1)
    rc = _load().orc_nm_check(_ptr(W, _i8p), n, k, N, M, ctypes.byref(br), ctypes.byref(bg))
    if rc == ERR_ARG:
        raise OracleError("nm_check: bad arguments")
    return rc == OK, br.value, bg.value


def pack_logical(W, N, M):
    """Canonical B_pack: (vals int8 [n, k/M, N], offs uint8 [n, k/M, N])."""
    W = _c(W, np.int8)
    n, k = W.shape
    vals = np.zeros((n, k // M, N), np.int8)
    offs = np.zeros((n, k // M, N), np.uint8)
    _check(_load().orc_pack_logical(_ptr(W, _i8p), n, k, N, M, _ptr(vals, _i8p), _ptr(offs, _u8p)),
           "pack_logical")
    return vals, offs


def unpack_logical(vals, offs, k, M):
    vals = _c(vals, np.int8)
    offs = _c(offs, np.uint8)
    n, G, N = vals.shape
    W = np.zeros((n, k), np.int8)
    _check(_load().orc_unpack_logical(_ptr(vals, _i8p), _ptr(offs, _u8p), n, k, N, M, _ptr(W, _i8p)),
           "unpack_logical")
    return W


def matmul_i8(X, W, nthreads=0):
    """Y = X W^T exactly (int64 accumulation, must fit int32)."""
    X = _c(X, np.int8)
    W = _c(W, np.int8)
    m, k = X.shape
    n, k2 = W.shape
    if k != k2:
        raise ValueError("reduction sizes differ")
    Y = np.zeros((m, n), np.int32)
    _check(_load().orc_matmul_i8(_ptr(X, _i8p), _ptr(W, _i8p), m, n, k, _ptr(Y, _i32p), nthreads),
           "matmul_i8")
    return Y


def matmul_i8_sampled(X, W, rows, cols):
    X = _c(X, np.int8)
    W = _c(W, np.int8)
    rows = _c(np.asarray(rows, np.int64), np.int64)
    cols = _c(np.asarray(cols, np.int64), np.int64)
    m, k = X.shape
    n = W.shape[0]
    out = np.zeros(rows.shape[0], np.int32)
    _check(_load().orc_matmul_i8_sampled(_ptr(X, _i8p), _ptr(W, _i8p), m, n, k, _ptr(rows, _i64p),
                                         _ptr(cols, _i64p), rows.shape[0], _ptr(out, _i32p)),
           "matmul_i8_sampled")
    return out


def spmm_packed(X, vals, offs, k, M, nthreads=0):
    X = _c(X, np.int8)
    vals = _c(vals, np.int8)
    offs = _c(offs, np.uint8)
    m = X.shape[0]
    n, G, N = vals.shape
    Y = np.zeros((m, n), np.int32)
    _check(_load().orc_spmm_packed(_ptr(X, _i8p), m, _ptr(vals, _i8p), _ptr(offs, _u8p), n, k, N, M,
                                   _ptr(Y, _i32p), nthreads), "spmm_packed")
    return Y


def f64_to_f16(x):
    """binary16 bit patterns (uint16) of float64 values, nearest-even."""
    x = _c(np.asarray(x, np.float64), np.float64)
    out = np.zeros(x.shape, np.uint16)
    _load().orc_f64_to_f16_array(_ptr(x, _f64p), x.size, _ptr(out, _u16p))
    return out


def dequant_f16(Y, scale):
    """binary16 bits of Y[i, j] * scale[j], computed in double, rounded once."""
    Y = _c(Y, np.int32)
    scale = _c(np.asarray(scale), np.float32)
    m, n = Y.shape
    out = np.zeros((m, n), np.uint16)
    _check(_load().orc_dequant_f16(_ptr(Y, _i32p), _ptr(scale, _f32p), m, n, _ptr(out, _u16p)),
           "dequant_f16")
    return out


def f16_to_f32(bits):
    """binary32 values of binary16 bit patterns (exact)."""
    bits = np.asarray(bits, np.uint16).ravel()
    return np.array([_load().orc_f16_to_f32(int(b)) for b in bits], np.float32)


def quantize_f16(xbits, inv_scale):
    """int8 codes of binary16 activations: q8(f32(x) * inv_scale), decided in binary32."""
    xbits = _c(np.asarray(xbits), np.uint16)
    out = np.zeros(xbits.shape, np.int8)
    _check(_load().orc_quantize_f16(_ptr(xbits, _u16p), xbits.size, ctypes.c_float(inv_scale),
                                    _ptr(out, _i8p)), "quantize_f16")
    return out


def requant_i8(Y, qscale):
    """int8 codes q8(f32(Y[i, j]) * qscale[j]), decided in binary32."""
    Y = _c(Y, np.int32)
    qscale = _c(np.asarray(qscale), np.float32)
    m, n = Y.shape
    out = np.zeros((m, n), np.int8)
    _check(_load().orc_requant_i8(_ptr(Y, _i32p), _ptr(qscale, _f32p), m, n, _ptr(out, _i8p)),
           "requant_i8")
    return out
