"""The C ABI library loads on a host without a GPU and exports every symbol
that the headers under include/ declare (no GPU compute call is made here)."""
import ctypes
import glob
import os
import re

from paper_2607_12505_amd import nmprobe, nmsearch, nmspmm

HEADERS = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                                        "*.h")))


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(nm_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def declared_in(header):
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(os.path.dirname(HEADERS[0]), header)).read(), flags=re.S)
    return set(re.findall(r"\b(nm_[a-z0-9_]+)\s*\(", src))


def test_header_declares_the_binding_names():
    assert len(HEADERS) == 3
    assert declared_functions() == sorted(nmspmm.EXPORTED + nmsearch.EXPORTED + nmprobe.EXPORTED)
    assert declared_in("nmprobe.h") == set(nmprobe.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = nmspmm.lib()
    for name in nmspmm.EXPORTED + nmsearch.EXPORTED:
        assert hasattr(lib, name), name
    probe = nmprobe.lib()
    for name in nmprobe.EXPORTED:
        assert hasattr(probe, name), name


def test_timing_event_calls_reject_null_pointers():
    # argument checks come before any runtime call, so they hold without a GPU
    import ctypes
    probe = nmprobe.lib()
    ms = ctypes.c_float()
    h = ctypes.c_void_p(1)
    assert probe.nm_probe_event_create(None) == nmspmm.NM_ERR_ARG
    assert probe.nm_probe_event_destroy(None) == nmspmm.NM_ERR_ARG
    assert probe.nm_probe_event_record(None, None) == nmspmm.NM_ERR_ARG
    assert probe.nm_probe_event_elapsed_ms(None, h, h) == nmspmm.NM_ERR_ARG
    assert probe.nm_probe_event_elapsed_ms(ctypes.byref(ms), None, h) == nmspmm.NM_ERR_ARG
    assert probe.nm_probe_event_elapsed_ms(ctypes.byref(ms), h, None) == nmspmm.NM_ERR_ARG


def test_method_library_carries_no_probe():
    # the measurement aids live in libnmprobe.so only
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", nmspmm.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    assert "nm_probe" not in out and "nm_wall_clock_khz" not in out


def test_one_hip_runtime_per_process():
    # the binding loads PyTorch's HIP runtime first, so the library binds to
    # it instead of starting a second one (which would find no device)
    nmspmm.lib()
    maps = open("/proc/self/maps").read().splitlines()
    runtimes = {line.split()[-1] for line in maps if "libamdhip64" in line}
    assert len(runtimes) == 1, runtimes


def test_expanded_descriptors():
    # every compact layout expands to the 2:4 layout or to a dense W of its shape
    for (N, M), sp in (((1, 4), True), ((1, 8), True), ((2, 8), True), ((3, 8), False), ((4, 8), False),
                       ((5, 8), False)):
        for n, k in ((64, 128), (200, 1040), (4, 16 * M)):
            d = nmspmm.compress_size(n, k, N, M)
            e, nbytes = nmspmm.expand_size(d)
            ref = nmspmm.compress_size(n, k, 2, 4) if sp else nmspmm.compress_size(n, k, 8, 8)
            assert e.layout == (nmspmm.NM_LAYOUT_SP42 if sp else nmspmm.NM_LAYOUT_DENSE)
            assert bytes(e) == bytes(ref)
            F, S = -(-n // 16), -(-k // 128)
            assert nbytes == (F * S * 1280 if sp else n * k)


def test_status_strings():
    for s in range(7):
        assert nmspmm.status_string(s)
    assert nmspmm.status_string(0) == "ok"
    assert nmspmm.status_string(99) == "unknown status"


def test_struct_sizes_match_header():
    # nm_desc: 8 int32 + 2 int64 + 2 int32 = 56 bytes; nm_plan: 8 int32 + 1 int64
    assert ctypes.sizeof(nmspmm.NmDesc) == 56
    assert ctypes.sizeof(nmspmm.NmPlan) == 40
    # nm_outputs: 5 pointers; nm_search_params: 4 int32 + 1 uint64
    assert ctypes.sizeof(nmspmm.NmOutputs) == 40
    assert ctypes.sizeof(nmsearch.NmSearchParams) == 24


def test_host_side_argument_checks_need_no_gpu():
    # These calls are rejected before any HIP call, so fake (aligned, non-null)
    # pointers are never dereferenced.
    L = nmspmm.lib()
    fake = ctypes.c_void_p(1 << 20)
    nul = ctypes.c_void_p(0)
    args = lambda m, n, Y, Yh: (fake, m, fake, n, 128, Y, fake, Yh, nul, 0, nul, None)
    assert L.nm_gemm_i8_dense_ex(*args(-1, 64, fake, nul)) == nmspmm.NM_ERR_SHAPE
    assert L.nm_gemm_i8_dense_ex(*args(0, 64, nul, nul)) == nmspmm.NM_OK           # m == 0: nothing examined
    assert L.nm_gemm_i8_dense_ex(*args(64, 64, nul, nul)) == nmspmm.NM_ERR_ARG     # no output
    assert L.nm_gemm_i8_dense_ex(*args(64, 66, fake, nul)) == nmspmm.NM_ERR_SHAPE  # n % 4 != 0
    # outputs are addressed with 32-bit byte offsets: m * n must stay below 2^29
    assert L.nm_gemm_i8_dense_ex(*args(1 << 20, 512, fake, nul)) == nmspmm.NM_ERR_SHAPE
    misaligned = ctypes.c_void_p((1 << 20) + 4)
    assert L.nm_gemm_i8_dense_ex(fake, 64, fake, 64, 128, misaligned, fake, nul, nul, 0, nul, None) == \
        nmspmm.NM_ERR_ARG
    o = nmspmm.NmOutputs(None, None, None, (1 << 20), None)                         # int8 output without qscale
    d = nmspmm.compress_size(64, 128, 2, 4)
    assert L.nm_spmm_out(fake, 64, fake, fake, ctypes.byref(d), ctypes.byref(o), nul, 0, nul, None) == \
        nmspmm.NM_ERR_ARG
    # expansion: only compact layouts, a large enough buffer, aligned pointers
    c28 = nmspmm.compress_size(64, 128, 2, 8)
    e, nbytes = nmspmm.NmDesc(), ctypes.c_size_t(0)
    for stored in (d, nmspmm.compress_size(64, 128, 8, 8)):                  # SP42 and DENSE
        assert L.nm_expand_size(ctypes.byref(stored), ctypes.byref(e), ctypes.byref(nbytes)) == nmspmm.NM_ERR_ARG
        assert L.nm_expand(ctypes.byref(stored), fake, fake, fake, 1 << 20, nul) == nmspmm.NM_ERR_ARG
    assert L.nm_expand_size(ctypes.byref(c28), None, ctypes.byref(nbytes)) == nmspmm.NM_ERR_ARG
    assert L.nm_expand(ctypes.byref(c28), fake, fake, fake, 64 * 1280 // 16 - 1, nul) == nmspmm.NM_ERR_WORKSPACE
    assert L.nm_expand(ctypes.byref(c28), fake, fake, misaligned, 1 << 20, nul) == nmspmm.NM_ERR_ARG
    assert L.nm_expand(ctypes.byref(c28), fake, nul, fake, 1 << 20, nul) == nmspmm.NM_ERR_ARG
    # a GEMM launch carrying an expansion: the job is checked before anything is launched
    y_out = nmspmm.NmOutputs(fake.value, None, None, None, None)
    job = nmspmm.NmExpandJob(ctypes.pointer(d), fake.value, fake.value, fake.value, 1 << 20)   # d is 2:4: stored form
    assert L.nm_spmm_out_expand(fake, 64, fake, fake, ctypes.byref(d), ctypes.byref(y_out), nul, 0, nul, None,
                                ctypes.byref(job)) == nmspmm.NM_ERR_ARG
    small = nmspmm.NmExpandJob(ctypes.pointer(c28), fake.value, fake.value, fake.value, 64)
    assert L.nm_gemm_i8_dense_out_expand(fake, 64, fake, 64, 128, ctypes.byref(y_out), nul, 0, nul, None,
                                         ctypes.byref(small)) == nmspmm.NM_ERR_WORKSPACE
    assert L.nm_gemm_i8_dense_out_expand(fake, -1, fake, 64, 128, ctypes.byref(y_out), nul, 0, nul, None,
                                         ctypes.byref(small)) == nmspmm.NM_ERR_SHAPE
    # the carried expansion may not write into anything the GEMM touches (checked before any launch)
    base = 1 << 30
    X, W, Yp = base, base + (1 << 24), base + (2 << 24)
    y_at = nmspmm.NmOutputs(Yp, None, None, None, None)
    for out_at in (X + 4096, W, Yp + 64 * 64 * 4 - 16):
        job = nmspmm.NmExpandJob(ctypes.pointer(c28), base + (3 << 24), base + (4 << 24), out_at, 1 << 16)
        assert L.nm_gemm_i8_dense_out_expand(ctypes.c_void_p(X), 64, ctypes.c_void_p(W), 64, 128, ctypes.byref(y_at),
                                             nul, 0, nul, None, ctypes.byref(job)) == nmspmm.NM_ERR_ARG
    assert L.nm_quantize_f16(fake, -1, ctypes.c_float(1.0), fake, nul) == nmspmm.NM_ERR_SHAPE
    assert L.nm_quantize_f16(misaligned, 16, ctypes.c_float(1.0), fake, nul) == nmspmm.NM_ERR_ARG
    P = nmprobe.lib()
    assert P.nm_probe_mfma_rate(nmspmm.NM_KIND_SP42, nul, 1, 1, fake, nul, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_rate(nmspmm.NM_KIND_C14, fake, 1, 1, fake, nul, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_rate(nmspmm.NM_KIND_DENSE, fake, 0, 1, fake, nul, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_rate(nmspmm.NM_KIND_DENSE, fake, 1, 0, fake, nul, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_wall_clock_khz(None) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_layout(nmspmm.NM_KIND_SP42, nul, fake, fake, fake, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_layout(nmspmm.NM_KIND_SP42, fake, fake, nul, fake, nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_mfma_layout(nmspmm.NM_KIND_C14, fake, fake, fake, fake, nul) == nmspmm.NM_ERR_ARG
    ok_plan = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 0, 1)
    y_only = nmspmm.NmOutputs(fake.value, None, None, None, None)
    assert P.nm_probe_store_only(None, 64, 64, ctypes.byref(y_only), nul) == nmspmm.NM_ERR_ARG
    assert P.nm_probe_store_only(ctypes.byref(ok_plan), 64, 66, ctypes.byref(y_only), nul) == nmspmm.NM_ERR_SHAPE
    assert P.nm_probe_store_only(ctypes.byref(ok_plan), -1, 64, ctypes.byref(y_only), nul) == nmspmm.NM_ERR_SHAPE
    assert P.nm_probe_store_only(ctypes.byref(ok_plan), 0, 64, ctypes.byref(y_only), nul) == nmspmm.NM_OK
    no_out = nmspmm.NmOutputs(None, None, None, None, None)
    assert P.nm_probe_store_only(ctypes.byref(ok_plan), 64, 64, ctypes.byref(no_out), nul) == nmspmm.NM_ERR_ARG
    fp16_no_scale = nmspmm.NmOutputs(None, fake.value, None, None, None)
    assert P.nm_probe_store_only(ctypes.byref(ok_plan), 64, 64, ctypes.byref(fp16_no_scale), nul) == nmspmm.NM_ERR_ARG
    for bad in (nmspmm.make_plan(nmspmm.NM_KIND_SP42, 10, 1),      # k-sliced layout
                nmspmm.make_plan(nmspmm.NM_KIND_SP42, 0, 2),       # split_k != 1
                nmspmm.make_plan(99, 0, 1)):                        # unknown kind
        assert P.nm_probe_store_only(ctypes.byref(bad), 64, 64, ctypes.byref(y_only), nul) == nmspmm.NM_ERR_ARG


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:  # pragma: no cover - torch is part of the image
        return False


def test_launch_failures_report_nm_err_hip():
    # Without a device every launch fails: each entry point must turn that into
    # NM_ERR_HIP (never a crash or NM_OK).  Skipped where a GPU is visible, since
    # the fake pointers below would then reach a real kernel.
    if _gpu_visible():
        import pytest
        pytest.skip("a GPU is visible: fake device pointers must not be launched")
    L = nmspmm.lib()
    fake, nul = ctypes.c_void_p(1 << 20), None
    d = nmspmm.compress_size(64, 128, 2, 4)
    assert L.nm_spmm_ex(fake, 64, fake, fake, ctypes.byref(d), fake, nul, nul, nul, 0, nul, None) == \
        nmspmm.NM_ERR_HIP
    assert L.nm_gemm_i8_dense_ex(fake, 64, fake, 64, 128, fake, nul, nul, nul, 0, nul, None) == nmspmm.NM_ERR_HIP
    assert L.nm_quantize_f16(fake, 16, ctypes.c_float(1.0), fake, nul) == nmspmm.NM_ERR_HIP
    assert L.nm_workspace_init(fake, 64, nul) == nmspmm.NM_ERR_HIP
    c14 = nmspmm.compress_size(64, 128, 1, 4)
    assert L.nm_expand(ctypes.byref(c14), fake, fake, fake, 1 << 20, nul) == nmspmm.NM_ERR_HIP
    y_out = nmspmm.NmOutputs(fake.value, None, None, None, None)
    far = [ctypes.c_void_p((1 << 32) + (i << 24)) for i in range(3)]    # the job's buffers, apart from the GEMM's
    job = nmspmm.NmExpandJob(ctypes.pointer(c14), far[0].value, far[1].value, far[2].value, 1 << 20)
    assert L.nm_spmm_out_expand(fake, 64, fake, fake, ctypes.byref(d), ctypes.byref(y_out), nul, 0, nul, None,
                                ctypes.byref(job)) == nmspmm.NM_ERR_HIP
    assert L.nm_gemm_i8_dense_out_expand(fake, 0, fake, 64, 128, ctypes.byref(y_out), nul, 0, nul, None,
                                         ctypes.byref(job)) == nmspmm.NM_ERR_HIP     # m == 0: the job alone
    P = nmprobe.lib()
    assert P.nm_probe_mfma_rate(nmspmm.NM_KIND_SP42, fake, 1, 1, fake, nul, nul) == nmspmm.NM_ERR_HIP
    khz = ctypes.c_int32(0)
    assert P.nm_wall_clock_khz(ctypes.byref(khz)) == nmspmm.NM_ERR_HIP
    assert P.nm_probe_mfma_layout(nmspmm.NM_KIND_DENSE, fake, fake, nul, fake, nul) == nmspmm.NM_ERR_HIP
    y_only = nmspmm.NmOutputs(fake.value, None, None, None, None)
    assert P.nm_probe_store_only(ctypes.byref(nmspmm.make_plan(nmspmm.NM_KIND_SP42, 0, 1)), 64, 64,
                                 ctypes.byref(y_only), nul) == nmspmm.NM_ERR_HIP
