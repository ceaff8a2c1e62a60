"""Thin ctypes binding of libnmspmm (C ABI in include/nmspmm.h).

Names follow the C entry points.  This module only marshals arguments: every
step of the GEMM runs in the library's HIP kernels.  PyTorch supplies device
memory and the current HIP stream; NumPy arrays carry host data for packing.
There is no fallback: if the library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import struct
import threading
import zlib
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnmspmm.so")

NM_OK, NM_ERR_ARG, NM_ERR_SHAPE, NM_ERR_PATTERN, NM_ERR_UNSUPPORTED, NM_ERR_WORKSPACE, NM_ERR_HIP = range(7)
NM_OUT_I32, NM_OUT_F16, NM_OUT_I8 = 1, 2, 4
NM_PLAN_EXPAND_CARRIED = 8
# kernel families; a packed layout and the family that consumes it share a number
NM_KIND_SP42, NM_KIND_C14, NM_KIND_DENSE, NM_KIND_C18, NM_KIND_C28, NM_KIND_MK3, NM_KIND_MK4, NM_KIND_MK5 = range(1, 9)
(NM_LAYOUT_SP42, NM_LAYOUT_C14, NM_LAYOUT_DENSE, NM_LAYOUT_C18, NM_LAYOUT_C28, NM_LAYOUT_MK3, NM_LAYOUT_MK4,
 NM_LAYOUT_MK5) = range(1, 9)
ALL_KINDS = tuple(range(1, 9))

# Every symbol the header declares (checked by the CPU tests).
EXPORTED = (
    "nm_status_string", "nm_compress_size", "nm_compress", "nm_decompress", "nm_num_tiles",
    "nm_tile_info", "nm_plan_kernel_name", "nm_spmm_plan", "nm_spmm_plan_complete", "nm_gemm_i8_dense_plan", "nm_workspace_size", "nm_workspace_init",
    "nm_spmm", "nm_spmm_ex", "nm_gemm_i8_dense", "nm_gemm_i8_dense_ex", "nm_spmm_out", "nm_gemm_i8_dense_out",
    "nm_quantize_f16", "nm_spmm_noalloc", "nm_expand_size", "nm_expand", "nm_spmm_out_expand",
    "nm_gemm_i8_dense_out_expand",
)
NM_NOALLOC_SCRATCH_BYTES = 16384 + (32 << 20)


class NmDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("nm_n", ctypes.c_int32), ("nm_m", ctypes.c_int32),
                ("kind", ctypes.c_int32), ("layout", ctypes.c_int32), ("n_frags", ctypes.c_int32),
                ("k_steps", ctypes.c_int32), ("vals_bytes", ctypes.c_int64), ("meta_bytes", ctypes.c_int64),
                ("bad_row", ctypes.c_int32), ("bad_group", ctypes.c_int32)]


class NmPlan(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("tile", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("tile_m", ctypes.c_int32), ("split_k", ctypes.c_int32), ("grid", ctypes.c_int32),
                ("expand", ctypes.c_int32), ("reserved", ctypes.c_int32), ("expand_bytes", ctypes.c_int64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class NmOutputs(ctypes.Structure):
    _fields_ = [("y", ctypes.c_void_p), ("yh", ctypes.c_void_p), ("scale", ctypes.c_void_p),
                ("yq", ctypes.c_void_p), ("qscale", ctypes.c_void_p)]


class NmExpandJob(ctypes.Structure):
    _fields_ = [("desc", ctypes.POINTER(NmDesc)), ("vals", ctypes.c_void_p), ("meta", ctypes.c_void_p),
                ("out", ctypes.c_void_p), ("out_bytes", ctypes.c_size_t)]


class NmError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """The loaded library.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_12505_amd/build.py")
        # PyTorch ships its own HIP runtime under the same soname as the
        # system one the library links.  Loaded first, it is the one the
        # library binds to, so a process has a single HIP runtime; loaded
        # after the library, a second runtime would start and find no device.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        pd, pp = ctypes.POINTER(NmDesc), ctypes.POINTER(NmPlan)
        sig = {
            "nm_status_string": ([i32], ctypes.c_char_p),
            "nm_compress_size": ([i32, i32, i32, i32, pd], i32),
            "nm_compress": ([vp, i32, i32, i32, i32, vp, vp, pd], i32),
            "nm_decompress": ([pd, vp, vp, vp], i32),
            "nm_num_tiles": ([], i32),
            "nm_tile_info": ([i32, ctypes.POINTER(i32), ctypes.POINTER(i32)], i32),
            "nm_plan_kernel_name": ([pp, ctypes.c_char_p, i32], i32),
            "nm_spmm_plan": ([pd, i32, i32, pp], i32),
            "nm_spmm_plan_complete": ([pd, i32, pp], i32),
            "nm_gemm_i8_dense_plan": ([i32, i32, i32, i32, pp], i32),
            "nm_workspace_size": ([pp, i32, i32, ctypes.POINTER(sz)], i32),
            "nm_workspace_init": ([vp, sz, vp], i32),
            "nm_spmm": ([vp, i32, vp, vp, pd, vp, vp, vp, vp, sz, vp], i32),
            "nm_spmm_ex": ([vp, i32, vp, vp, pd, vp, vp, vp, vp, sz, vp, pp], i32),
            "nm_gemm_i8_dense": ([vp, i32, vp, i32, i32, vp, vp, vp, vp, sz, vp], i32),
            "nm_gemm_i8_dense_ex": ([vp, i32, vp, i32, i32, vp, vp, vp, vp, sz, vp, pp], i32),
            "nm_spmm_out": ([vp, i32, vp, vp, pd, ctypes.POINTER(NmOutputs), vp, sz, vp, pp], i32),
            "nm_gemm_i8_dense_out": ([vp, i32, vp, i32, i32, ctypes.POINTER(NmOutputs), vp, sz, vp, pp], i32),
            "nm_quantize_f16": ([vp, ctypes.c_int64, ctypes.c_float, vp, vp], i32),
            "nm_spmm_noalloc": ([vp, i32, vp, vp, pd, ctypes.POINTER(NmOutputs), vp, pp], i32),
            "nm_expand_size": ([pd, pd, ctypes.POINTER(sz)], i32),
            "nm_expand": ([pd, vp, vp, vp, sz, vp], i32),
            "nm_spmm_out_expand": ([vp, i32, vp, vp, pd, ctypes.POINTER(NmOutputs), vp, sz, vp, pp,
                                    ctypes.POINTER(NmExpandJob)], i32),
            "nm_gemm_i8_dense_out_expand": ([vp, i32, vp, i32, i32, ctypes.POINTER(NmOutputs), vp, sz, vp, pp,
                                             ctypes.POINTER(NmExpandJob)], i32),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
        return L


def status_string(status: int) -> str:
    return lib().nm_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != NM_OK:
        raise NmError(status, what)


# ---------------------------------------------------------------- packing (host)

@dataclasses.dataclass
class Packed:
    """Host result of nm_compress: packed values, packed positions, descriptor."""
    vals: np.ndarray
    meta: np.ndarray
    desc: NmDesc


# ---------------------------------------------------------------------------
# Packed-weight files: nm_compress runs once offline, so its output is kept on
# disk.  Layout (little-endian): 8-byte magic, u32 version, u32 header bytes,
# the descriptor's fields (8 x i32: n, k, nm_n, nm_m, kind, layout,
# n_frags, k_steps; 2 x i64: vals_bytes, meta_bytes), CRC-32 of the values
# and of the positions (2 x u32), then the values and the positions.

PACKED_MAGIC = b"NMSPMM\x00\x01"
PACKED_VERSION = 2
_PACKED_HEAD = struct.Struct("<8sII8i2q2I")


def save_packed(path: str, p: "Packed") -> None:
    d = p.desc
    vals, meta = np.ascontiguousarray(p.vals).view(np.uint8), np.ascontiguousarray(p.meta).view(np.uint8)
    if vals.size != d.vals_bytes or meta.size != d.meta_bytes:
        raise ValueError("packed arrays do not match their descriptor")
    head = _PACKED_HEAD.pack(PACKED_MAGIC, PACKED_VERSION, _PACKED_HEAD.size, d.n, d.k, d.nm_n, d.nm_m, d.kind,
                             d.layout, d.n_frags, d.k_steps, d.vals_bytes, d.meta_bytes,
                             zlib.crc32(vals.tobytes()), zlib.crc32(meta.tobytes()))
    with open(path, "wb") as f:
        f.write(head)
        f.write(vals.tobytes())
        f.write(meta.tobytes())


def load_packed(path: str) -> "Packed":
    """Reads a file written by save_packed.  The descriptor is checked against
    the library's own nm_compress_size of (n, k, N, M) and both checksums are
    verified; any mismatch raises ValueError."""
    with open(path, "rb") as f:
        raw = f.read()
    if len(raw) < _PACKED_HEAD.size:
        raise ValueError(f"{path}: truncated header")
    (magic, version, hsize, n, k, nm_n, nm_m, kind, layout, n_frags, k_steps, vb, mb, cv,
     cm) = _PACKED_HEAD.unpack_from(raw)
    if magic != PACKED_MAGIC or version != PACKED_VERSION or hsize != _PACKED_HEAD.size:
        raise ValueError(f"{path}: not a packed-weight file of version {PACKED_VERSION}")
    want = compress_size(n, k, nm_n, nm_m)
    got = (kind, layout, n_frags, k_steps, vb, mb)
    if got != (want.kind, want.layout, want.n_frags, want.k_steps, want.vals_bytes, want.meta_bytes):
        raise ValueError(f"{path}: descriptor does not match nm_compress_size({n}, {k}, {nm_n}, {nm_m})")
    if len(raw) != hsize + vb + mb:
        raise ValueError(f"{path}: {len(raw)} bytes, expected {hsize + vb + mb}")
    vals = np.frombuffer(raw, dtype=np.int8, count=vb, offset=hsize).copy()
    meta = np.frombuffer(raw, dtype=np.uint8, count=mb, offset=hsize + vb).copy()
    if zlib.crc32(vals.view(np.uint8).tobytes()) != cv or zlib.crc32(meta.tobytes()) != cm:
        raise ValueError(f"{path}: checksum mismatch")
    return Packed(vals, meta, want)


def compress_size(n: int, k: int, N: int, M: int) -> NmDesc:
    d = NmDesc()
    _check(lib().nm_compress_size(n, k, N, M, ctypes.byref(d)), "nm_compress_size")
    return d


def compress(W: np.ndarray, N: int, M: int) -> Packed:
    W = np.ascontiguousarray(W)
    if W.dtype != np.int8 or W.ndim != 2:
        raise TypeError("W must be a 2-D int8 array")
    n, k = W.shape
    d = NmDesc()
    st = lib().nm_compress_size(n, k, N, M, ctypes.byref(d))
    if st != NM_OK:
        raise NmError(st, "nm_compress")
    vals = np.empty(d.vals_bytes, np.int8)
    meta = np.empty(d.meta_bytes, np.uint8)
    st = lib().nm_compress(W.ctypes.data, n, k, N, M, vals.ctypes.data, meta.ctypes.data, ctypes.byref(d))
    if st != NM_OK:
        err = NmError(st, "nm_compress")
        err.bad_row, err.bad_group = d.bad_row, d.bad_group
        raise err
    return Packed(vals, meta, d)


def decompress(p: Packed) -> np.ndarray:
    W = np.empty((p.desc.n, p.desc.k), np.int8)
    vals = np.ascontiguousarray(p.vals)
    meta = np.ascontiguousarray(p.meta)
    _check(lib().nm_decompress(ctypes.byref(p.desc), vals.ctypes.data, meta.ctypes.data, W.ctypes.data),
           "nm_decompress")
    return W


# ---------------------------------------------------------------- planning

def num_tiles() -> int:
    return lib().nm_num_tiles()


def tile_info(tile: int):
    a, b = ctypes.c_int(), ctypes.c_int()
    _check(lib().nm_tile_info(tile, ctypes.byref(a), ctypes.byref(b)), "nm_tile_info")
    return a.value, b.value


def plan_kernel_name(plan: NmPlan) -> str:
    buf = ctypes.create_string_buffer(128)
    _check(lib().nm_plan_kernel_name(ctypes.byref(plan), buf, 128), "nm_plan_kernel_name")
    return buf.value.decode()


def spmm_plan(desc: NmDesc, m: int, out_mode: int = NM_OUT_I32) -> NmPlan:
    p = NmPlan()
    _check(lib().nm_spmm_plan(ctypes.byref(desc), m, out_mode, ctypes.byref(p)), "nm_spmm_plan")
    return p


def spmm_plan_complete(desc: NmDesc, m: int, plan: NmPlan) -> NmPlan:
    """nm_spmm_plan_complete: a copy of a caller-built plan with the library's fields filled."""
    p = NmPlan.from_buffer_copy(plan)
    _check(lib().nm_spmm_plan_complete(ctypes.byref(desc), m, ctypes.byref(p)), "nm_spmm_plan_complete")
    return p


def dense_plan(m: int, n: int, k: int, out_mode: int = NM_OUT_I32) -> NmPlan:
    p = NmPlan()
    _check(lib().nm_gemm_i8_dense_plan(m, n, k, out_mode, ctypes.byref(p)), "nm_gemm_i8_dense_plan")
    return p


def make_plan(kind: int, tile: int, split_k: int, expand: int = 0) -> NmPlan:
    p = NmPlan()
    p.kind, p.tile, p.split_k, p.expand = kind, tile, split_k, expand
    return p


def workspace_size(plan: NmPlan, m: int, n: int) -> int:
    b = ctypes.c_size_t()
    _check(lib().nm_workspace_size(ctypes.byref(plan), m, n, ctypes.byref(b)), "nm_workspace_size")
    return b.value


# ---------------------------------------------------------------- device side (torch for memory/streams)

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Workspace:
    """A zero-initialised device buffer that grows on demand (one per device).

    The library keeps its counters at zero after every call, so the buffer is
    initialised once, when it is (re)allocated."""

    def __init__(self):
        self._bufs = {}

    def get(self, nbytes: int, device):
        torch = _torch()
        if nbytes == 0:
            return None, 0
        key = torch.device(device).index or 0
        buf = self._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.zeros(max(nbytes, 1 << 20), dtype=torch.uint8, device=device)
            self._bufs[key] = buf
        return buf, buf.numel()


_WS = Workspace()


@dataclasses.dataclass
class DeviceWeight:
    """A packed weight resident on the GPU (values, positions, host descriptor)."""
    vals: object
    meta: object
    desc: NmDesc

    @classmethod
    def from_packed(cls, p: Packed, device="cuda"):
        torch = _torch()
        v = torch.from_numpy(p.vals).to(device)
        m = torch.from_numpy(p.meta).to(device)
        return cls(v, m, p.desc)


def _need(t, name, dtypes, shape=None, numel=None):
    """Validates one tensor argument before its address reaches the library:
    the C ABI takes bare pointers, so a tensor of the wrong size, type or
    layout would otherwise be read or written out of bounds on the GPU."""
    if t is None:
        return
    if t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype}, expected one of {[str(d) for d in dtypes]}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {numel} needed")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def _on_device(named, device=None):
    """Every given tensor is a device tensor, all on one device."""
    for name, t in named:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name}: must be a device tensor")
        if device is None:
            device = t.device
        elif t.device != device:
            raise ValueError(f"{name}: on {t.device}, expected {device}")


def _check_outputs(torch, m, n, Y, scale, Yh, Yq, qscale):
    _need(Y, "Y", (torch.int32,), (m, n))
    _need(Yh, "Yh", (torch.float16, torch.int16), (m, n))
    _need(Yq, "Yq", (torch.int8,), (m, n))
    _need(scale, "scale", (torch.float32,), (n,))
    _need(qscale, "qscale", (torch.float32,), (n,))


_WS_DTYPES = ("uint8", "int8", "int32", "int64", "float32")


def _check_ws(torch, ws):
    _need(ws, "ws", tuple(getattr(torch, d) for d in _WS_DTYPES))


def _outputs(Y, scale, Yh, Yq, qscale) -> NmOutputs:
    return NmOutputs(_ptr(Y), _ptr(Yh), _ptr(scale), _ptr(Yq), _ptr(qscale))


def _out_mode(Y, Yh, Yq) -> int:
    mode = (NM_OUT_I32 if Y is not None else 0) | (NM_OUT_F16 if Yh is not None else 0)
    return mode | (NM_OUT_I8 if Yq is not None else 0)


def spmm(X, w: DeviceWeight, Y=None, scale=None, Yh=None, plan: Optional[NmPlan] = None, ws=None,
         stream=None, Yq=None, qscale=None, job: Optional[NmExpandJob] = None):
    """Sparse GEMM on torch device tensors.  Y (int32), Yh (float16, or int16
    view of binary16) and Yq (int8) are written in place; returns (Y, Yh), or
    (Y, Yh, Yq) when Yq is given.  Without Yq this calls nm_spmm_ex, with it
    nm_spmm_out; with an expansion job (expand_job()) nm_spmm_out_expand."""
    torch = _torch()
    d = w.desc
    if X.dim() != 2:
        raise ValueError(f"X: {X.dim()}-D, expected [m x {d.k}]")
    m = X.shape[0]
    _need(X, "X", (torch.int8,), (m, d.k))
    _need(w.vals, "w.vals", (torch.int8,), numel=d.vals_bytes)
    _need(w.meta, "w.meta", (torch.uint8,), numel=d.meta_bytes)
    _check_outputs(torch, m, d.n, Y, scale, Yh, Yq, qscale)
    _check_ws(torch, ws)
    _on_device((("X", X), ("w.vals", w.vals), ("w.meta", w.meta), ("Y", Y), ("Yh", Yh), ("Yq", Yq),
                ("scale", scale), ("qscale", qscale), ("ws", ws)))
    mode = _out_mode(Y, Yh, Yq)
    p = spmm_plan_complete(w.desc, m, plan) if plan is not None else spmm_plan(w.desc, m, mode or NM_OUT_I32)
    need = workspace_size(p, m, w.desc.n)
    if ws is None:
        ws, ws_bytes = _WS.get(need, X.device)
    else:
        ws_bytes = ws.numel() * ws.element_size()
    pl = ctypes.byref(plan) if plan is not None else None
    if job is not None:
        o = _outputs(Y, scale, Yh, Yq, qscale)
        st = lib().nm_spmm_out_expand(_ptr(X), m, _ptr(w.vals), _ptr(w.meta), ctypes.byref(w.desc), ctypes.byref(o),
                                      _ptr(ws), ws_bytes, _stream(stream), pl, ctypes.byref(job))
        _check(st, "nm_spmm_out_expand")
        return (Y, Yh) if Yq is None and qscale is None else (Y, Yh, Yq)
    if Yq is None and qscale is None:
        st = lib().nm_spmm_ex(_ptr(X), m, _ptr(w.vals), _ptr(w.meta), ctypes.byref(w.desc), _ptr(Y), _ptr(scale),
                              _ptr(Yh), _ptr(ws), ws_bytes, _stream(stream), pl)
        _check(st, "nm_spmm")
        return Y, Yh
    o = _outputs(Y, scale, Yh, Yq, qscale)
    st = lib().nm_spmm_out(_ptr(X), m, _ptr(w.vals), _ptr(w.meta), ctypes.byref(w.desc), ctypes.byref(o), _ptr(ws),
                           ws_bytes, _stream(stream), pl)
    _check(st, "nm_spmm_out")
    return Y, Yh, Yq


def spmm_noalloc(X, w: DeviceWeight, Y=None, scale=None, Yh=None, Yq=None, qscale=None,
                 plan: Optional[NmPlan] = None, stream=None):
    """nm_spmm_noalloc: nm_spmm_out with the library's static scratch in place
    of a workspace (nothing is allocated by the call).  Returns (Y, Yh, Yq)."""
    torch = _torch()
    d = w.desc
    if X.dim() != 2:
        raise ValueError(f"X: {X.dim()}-D, expected [m x {d.k}]")
    m = X.shape[0]
    _need(X, "X", (torch.int8,), (m, d.k))
    _need(w.vals, "w.vals", (torch.int8,), numel=d.vals_bytes)
    _need(w.meta, "w.meta", (torch.uint8,), numel=d.meta_bytes)
    _check_outputs(torch, m, d.n, Y, scale, Yh, Yq, qscale)
    _on_device((("X", X), ("w.vals", w.vals), ("w.meta", w.meta), ("Y", Y), ("Yh", Yh), ("Yq", Yq),
                ("scale", scale), ("qscale", qscale)))
    o = _outputs(Y, scale, Yh, Yq, qscale)
    pl = ctypes.byref(plan) if plan is not None else None
    _check(lib().nm_spmm_noalloc(_ptr(X), m, _ptr(w.vals), _ptr(w.meta), ctypes.byref(d), ctypes.byref(o),
                                 _stream(stream), pl), "nm_spmm_noalloc")
    return Y, Yh, Yq


def gemm_i8_dense(X, W, Y=None, scale=None, Yh=None, plan: Optional[NmPlan] = None, ws=None, stream=None,
                  Yq=None, qscale=None, job: Optional[NmExpandJob] = None):
    """Dense baseline GEMM (nm_gemm_i8_dense_ex, or nm_gemm_i8_dense_out when Yq is given, or
    nm_gemm_i8_dense_out_expand with an expansion job)."""
    torch = _torch()
    if X.dim() != 2 or W.dim() != 2:
        raise ValueError("X and W must be 2-D ([m x k] and [n x k])")
    m, k = X.shape
    n = W.shape[0]
    _need(X, "X", (torch.int8,), (m, k))
    _need(W, "W", (torch.int8,), (n, k))
    _check_outputs(torch, m, n, Y, scale, Yh, Yq, qscale)
    _check_ws(torch, ws)
    _on_device((("X", X), ("W", W), ("Y", Y), ("Yh", Yh), ("Yq", Yq), ("scale", scale), ("qscale", qscale),
                ("ws", ws)))
    mode = _out_mode(Y, Yh, Yq)
    p = plan if plan is not None else dense_plan(m, n, k, mode or NM_OUT_I32)
    need = workspace_size(p, m, n)
    if ws is None:
        ws, ws_bytes = _WS.get(need, X.device)
    else:
        ws_bytes = ws.numel() * ws.element_size()
    pl = ctypes.byref(plan) if plan is not None else None
    if job is not None:
        o = _outputs(Y, scale, Yh, Yq, qscale)
        st = lib().nm_gemm_i8_dense_out_expand(_ptr(X), m, _ptr(W), n, k, ctypes.byref(o), _ptr(ws), ws_bytes,
                                               _stream(stream), pl, ctypes.byref(job))
        _check(st, "nm_gemm_i8_dense_out_expand")
        return (Y, Yh) if Yq is None and qscale is None else (Y, Yh, Yq)
    if Yq is None and qscale is None:
        st = lib().nm_gemm_i8_dense_ex(_ptr(X), m, _ptr(W), n, k, _ptr(Y), _ptr(scale), _ptr(Yh), _ptr(ws),
                                       ws_bytes, _stream(stream), pl)
        _check(st, "nm_gemm_i8_dense")
        return Y, Yh
    o = _outputs(Y, scale, Yh, Yq, qscale)
    st = lib().nm_gemm_i8_dense_out(_ptr(X), m, _ptr(W), n, k, ctypes.byref(o), _ptr(ws), ws_bytes,
                                    _stream(stream), pl)
    _check(st, "nm_gemm_i8_dense_out")
    return Y, Yh, Yq


def expand_size(desc: NmDesc):
    """nm_expand_size: (descriptor of the expanded weight, bytes of its buffer)."""
    e = NmDesc()
    nbytes = ctypes.c_size_t(0)
    _check(lib().nm_expand_size(ctypes.byref(desc), ctypes.byref(e), ctypes.byref(nbytes)), "nm_expand_size")
    return e, nbytes.value


def expand(w: DeviceWeight, out=None, stream=None) -> DeviceWeight:
    """nm_expand: the compact weight w expanded (2:4 layout or dense W) into
    out (a uint8 or int8 device buffer of at least expand_size() bytes; one is
    allocated when None).  Returns a DeviceWeight of the expanded descriptor
    whose vals and meta are views of out."""
    torch = _torch()
    d = w.desc
    e, nbytes = expand_size(d)
    _need(w.vals, "w.vals", (torch.int8,), numel=d.vals_bytes)
    _need(w.meta, "w.meta", (torch.uint8,), numel=d.meta_bytes)
    if out is None:
        out = torch.empty(nbytes, dtype=torch.uint8, device=w.vals.device)
    _need(out, "out", (torch.uint8, torch.int8), numel=nbytes)
    if out.dim() != 1:
        raise ValueError("out: must be 1-D")
    _on_device((("w.vals", w.vals), ("w.meta", w.meta), ("out", out)))
    _check(lib().nm_expand(ctypes.byref(d), _ptr(w.vals), _ptr(w.meta), _ptr(out), out.numel(), _stream(stream)),
           "nm_expand")
    return _expanded_view(out, e)


def _expanded_view(out, e):
    torch = _torch()
    b = out.view(torch.uint8)
    return DeviceWeight(b[:e.vals_bytes].view(torch.int8), b[e.vals_bytes:e.vals_bytes + e.meta_bytes], e)


def expand_job(w: DeviceWeight, out):
    """An nm_expand_job for a GEMM launch to carry: w expanded into out (a
    uint8 or int8 device buffer of at least expand_size() bytes).  Returns
    (job, expanded DeviceWeight viewing out); keep both alive until the launch
    has run."""
    torch = _torch()
    d = w.desc
    e, nbytes = expand_size(d)
    _need(w.vals, "w.vals", (torch.int8,), numel=d.vals_bytes)
    _need(w.meta, "w.meta", (torch.uint8,), numel=d.meta_bytes)
    _need(out, "out", (torch.uint8, torch.int8), numel=nbytes)
    if out.dim() != 1:
        raise ValueError("out: must be 1-D")
    _on_device((("w.vals", w.vals), ("w.meta", w.meta), ("out", out)))
    job = NmExpandJob(ctypes.pointer(d), _ptr(w.vals), _ptr(w.meta), _ptr(out), out.numel())
    return job, _expanded_view(out, e)


def quantize_f16(x, inv_scale: float, xq=None, stream=None):
    """nm_quantize_f16: int8 codes of a float16 (or int16-bits) device tensor."""
    torch = _torch()
    _need(x, "x", (torch.float16, torch.int16))
    if xq is None:
        xq = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    _need(xq, "xq", (torch.int8,), tuple(x.shape))
    _on_device((("x", x), ("xq", xq)))
    _check(lib().nm_quantize_f16(_ptr(x), x.numel(), float(inv_scale), _ptr(xq), _stream(stream)),
           "nm_quantize_f16")
    return xq


def workspace_init(ws, stream=None):
    _check_ws(_torch(), ws)
    _on_device((("ws", ws),))
    _check(lib().nm_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "nm_workspace_init")
