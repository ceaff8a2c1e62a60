"""Thin ctypes binding of libnmprobe (C ABI in include/nmprobe.h): measurement
and test aids beside the method -- the matrix-instruction rate loop, the
single-instruction layout probe and the store-only run of a GEMM plan.

Only marshals arguments; PyTorch supplies device memory and the current HIP
stream.  The library links libnmspmm, which is loaded first."""
from __future__ import annotations

import ctypes
import os
import threading

from . import nmspmm
from .nmspmm import NM_KIND_DENSE, NM_KIND_SP42, NmOutputs, NmPlan, _check, _check_outputs, _on_device, _outputs
from .nmspmm import _ptr, _stream, _torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libnmprobe.so")

# Every symbol include/nmprobe.h declares (checked by the CPU tests).
EXPORTED = ("nm_probe_mfma_rate", "nm_probe_mfma_layout", "nm_wall_clock_khz", "nm_probe_store_only",
            "nm_probe_event_create", "nm_probe_event_destroy", "nm_probe_event_record", "nm_probe_event_elapsed_ms")
NM_PROBE_WORDS = 4096

_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """The loaded probe library.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_12505_amd/build.py")
        nmspmm.lib()  # PyTorch's HIP runtime and the method's library first
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int
        sig = {
            "nm_probe_mfma_rate": ([i32, vp, i32, i32, vp, vp, vp], i32),
            "nm_wall_clock_khz": ([ctypes.POINTER(ctypes.c_int32)], i32),
            "nm_probe_mfma_layout": ([i32, vp, vp, vp, vp, vp], i32),
            "nm_probe_store_only": ([ctypes.POINTER(NmPlan), i32, i32, ctypes.POINTER(NmOutputs), vp], i32),
            "nm_probe_event_create": ([ctypes.POINTER(vp)], i32),
            "nm_probe_event_destroy": ([vp], i32),
            "nm_probe_event_record": ([vp, vp], i32),
            "nm_probe_event_elapsed_ms": ([ctypes.POINTER(ctypes.c_float), vp, vp], i32),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
        return L


def probe_mfma_rate(kind: int, operands, iters: int, out, ticks=None, stream=None):
    """nm_probe_mfma_rate: launches the matrix-instruction rate loop.

    operands: int32 device tensor of NM_PROBE_WORDS words; out: int32 device
    tensor whose size (a multiple of 256) sets the number of workgroups;
    ticks: optional int64 device tensor of 2 words per workgroup."""
    wgs = out.numel() // 256
    if operands.numel() < NM_PROBE_WORDS or out.numel() % 256 or (ticks is not None and ticks.numel() < 2 * wgs):
        raise ValueError("operands needs NM_PROBE_WORDS words, out a multiple of 256, ticks 2 per workgroup")
    _check(lib().nm_probe_mfma_rate(int(kind), _ptr(operands), int(iters), wgs, _ptr(out), _ptr(ticks),
                                    _stream(stream)), "nm_probe_mfma_rate")


def wall_clock_khz() -> int:
    """nm_wall_clock_khz: rate of the device's real-time counter."""
    khz = ctypes.c_int32(0)
    _check(lib().nm_wall_clock_khz(ctypes.byref(khz)), "nm_wall_clock_khz")
    return int(khz.value)


def probe_mfma_layout(kind: int, a, b, pos, d, stream=None):
    """nm_probe_mfma_layout: one matrix instruction on one wave.

    a, d: int32 device tensors of 256 words; b: 512 words (NM_KIND_SP42) or
    256 (NM_KIND_DENSE); pos: 64 words (NM_KIND_SP42) or None."""
    nb = 512 if kind == NM_KIND_SP42 else 256
    if a.numel() < 256 or d.numel() < 256 or b.numel() < nb or (kind == NM_KIND_SP42 and
                                                                 (pos is None or pos.numel() < 64)):
        raise ValueError("operand buffers smaller than the instruction needs")
    _check(lib().nm_probe_mfma_layout(int(kind), _ptr(a), _ptr(b), _ptr(pos), _ptr(d), _stream(stream)),
           "nm_probe_mfma_layout")


def probe_store_only(plan: NmPlan, m: int, n: int, Y=None, scale=None, Yh=None, Yq=None, qscale=None, stream=None):
    """nm_probe_store_only: the plan's kernel with the reduction skipped, so
    only its epilogue stores run; the outputs receive zeros."""
    torch = _torch()
    _check_outputs(torch, m, n, Y, scale, Yh, Yq, qscale)
    _on_device((("Y", Y), ("Yh", Yh), ("Yq", Yq), ("scale", scale), ("qscale", qscale)))
    o = _outputs(Y, scale, Yh, Yq, qscale)
    _check(lib().nm_probe_store_only(ctypes.byref(plan), int(m), int(n), ctypes.byref(o), _stream(stream)),
           "nm_probe_store_only")


__all__ = ["EXPORTED", "NM_PROBE_WORDS", "NM_KIND_DENSE", "NM_KIND_SP42", "lib", "probe_mfma_rate",
           "wall_clock_khz", "probe_mfma_layout", "probe_store_only"]


class TimingEvent:
    """A fence-free timing event (nm_probe_event_*), with the record /
    elapsed_time interface of torch.cuda.Event(enable_timing=True)."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(lib().nm_probe_event_create(ctypes.byref(h)), "nm_probe_event_create")
        self._h = h

    def record(self, stream=None):
        _check(lib().nm_probe_event_record(self._h, _stream(stream)), "nm_probe_event_record")

    def elapsed_time(self, end: "TimingEvent") -> float:
        ms = ctypes.c_float()
        _check(lib().nm_probe_event_elapsed_ms(ctypes.byref(ms), self._h, end._h), "nm_probe_event_elapsed_ms")
        return float(ms.value)

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.nm_probe_event_destroy(h)
