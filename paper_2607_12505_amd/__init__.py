"""N:M sparse INT8 GEMM for AMD Instinct MI355X (gfx950).

The compute lives in ``libnmspmm.so`` (hand-written HIP kernels behind a C
ABI, declared in ``include/nmspmm.h``).  ``paper_2607_12505_amd.nmspmm`` is the
thin ctypes binding; importing this package does not load the library.
"""
__all__ = ["nmspmm", "workloads"]
