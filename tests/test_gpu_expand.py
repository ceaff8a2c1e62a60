"""nm_expand (the decode of a compact weight as a pass of its own, Sec. 4.2)
through the C ABI, alone and carried by a GEMM launch: the expanded buffer,
read by the header's formulas, holds exactly the weight that was packed; the
GEMM on the expanded descriptor gives the oracle's product bit for bit;
nothing is written past the buffer, and an undersized buffer is rejected
before anything is written."""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl

from gpu_util import run_sparse

pytestmark = pytest.mark.gpu

COMPACT = ((1, 4), (1, 8), (2, 8), (3, 8), (4, 8), (5, 8))
SHAPES = ((64, 128), (200, 1040), (52, 256), (4, 16 * 8))
SENTINEL = 0xA5
GUARD = 4096


def effective_weight_sp42(buf, e):
    """The weight the structured-sparse instruction multiplies with, from a
    2:4-layout buffer (values then positions) read by the header's formulas:
    every slot adds its value at its position (padding slots hold zeros)."""
    F, S = e.n_frags, e.k_steps
    v = buf[:e.vals_bytes].view(np.int8).reshape(F, S, 64, 8, 2).astype(np.int64)
    w = buf[e.vals_bytes:e.vals_bytes + e.meta_bytes].view(np.uint32).reshape(F, S, 64).astype(np.int64)
    f, s, lane, g, t = np.meshgrid(np.arange(F), np.arange(S), np.arange(64), np.arange(8), np.arange(2),
                                   indexing="ij")
    pos = (w[f, s, lane] >> (4 * g + 2 * t)) & 3
    rows = 16 * f + lane % 16
    cols = 128 * s + 32 * (lane // 16) + 4 * g + pos
    Wr = np.zeros((16 * F, 128 * S), np.int64)
    np.add.at(Wr, (rows.ravel(), cols.ravel()), v.ravel())
    return Wr


def expand_on_device(packed, nbytes_extra=GUARD):
    import torch
    e, nbytes = nmspmm.expand_size(packed.desc)
    dw = nmspmm.DeviceWeight.from_packed(packed)
    out = torch.full((nbytes + nbytes_extra,), SENTINEL, dtype=torch.uint8, device="cuda")
    ew = nmspmm.expand(dw, out=out)
    torch.cuda.synchronize()
    h = out.cpu().numpy()
    assert (h[nbytes:] == SENTINEL).all(), "write past the expanded weight"
    return e, h[:nbytes], ew


@pytest.mark.parametrize("N,M", COMPACT)
@pytest.mark.parametrize("n,k", SHAPES)
def test_expanded_weight_is_the_packed_weight(N, M, n, k):
    rng = np.random.default_rng(1000 * N + M + n + k)
    for full in (True, False):
        W = wl.random_nm(n, k, N, M, rng, full=full)
        packed = nmspmm.compress(W, N, M)
        e, h, _ = expand_on_device(packed)
        if e.layout == nmspmm.NM_LAYOUT_DENSE:
            assert np.array_equal(h.view(np.int8).reshape(n, k), W)
        else:
            Wr = effective_weight_sp42(h, e)
            assert np.array_equal(Wr[:n, :k], W.astype(np.int64))
            assert not Wr[n:].any() and not Wr[:, k:].any()
            # the 4:2 operand holds at most 2 nonzeros per 4-group by construction
            vals = h[:e.vals_bytes].view(np.int8).reshape(-1, 8, 2)
            assert vals.shape[0] == e.n_frags * e.k_steps * 64


@pytest.mark.parametrize("N,M", COMPACT)
def test_gemm_on_expanded_weight_matches_oracle(N, M):
    import torch
    rng = np.random.default_rng(77 + N * M)
    m, n, k = 333, 200, 1040
    X = rng.integers(-128, 128, (m, k), dtype=np.int64).astype(np.int8)
    W = wl.random_nm(n, k, N, M, rng, full=True)
    packed = nmspmm.compress(W, N, M)
    ref = oracle.matmul_i8(X, W)
    _, _, ew = expand_on_device(packed)
    Xd = torch.from_numpy(X).cuda()
    Y = torch.full((m, n), -7, dtype=torch.int32, device="cuda")
    nmspmm.spmm(Xd, ew, Y=Y)
    torch.cuda.synchronize()
    assert np.array_equal(Y.cpu().numpy(), ref)
    # and the same as the GEMM on the compact weight, with its own plan
    Yc, _ = run_sparse(X, packed)
    assert np.array_equal(Yc, ref)


def test_undersized_buffer_is_rejected_untouched():
    import torch
    rng = np.random.default_rng(5)
    W = wl.random_nm(64, 256, 2, 8, rng, full=True)
    packed = nmspmm.compress(W, 2, 8)
    _, nbytes = nmspmm.expand_size(packed.desc)
    dw = nmspmm.DeviceWeight.from_packed(packed)
    out = torch.full((nbytes - 16,), SENTINEL, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):
        nmspmm.expand(dw, out=out)
    import ctypes
    st = nmspmm.lib().nm_expand(ctypes.byref(packed.desc), dw.vals.data_ptr(), dw.meta.data_ptr(), out.data_ptr(),
                                out.numel(), None)
    assert st == nmspmm.NM_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == SENTINEL).all()


def test_stored_layouts_are_rejected():
    rng = np.random.default_rng(6)
    for N, M in ((2, 4), (8, 8)):
        packed = nmspmm.compress(wl.random_nm(32, 128, N, M, rng), N, M)
        with pytest.raises(nmspmm.NmError):
            nmspmm.expand(nmspmm.DeviceWeight.from_packed(packed))


# ---------------------------------------------------------------------------
# GEMM launches that carry an expansion (nm_spmm_out_expand,
# nm_gemm_i8_dense_out_expand): the GEMM's outputs are the oracle's product,
# the carried expansion is byte-identical to nm_expand's, nothing is written
# past either, for GEMMs on every kernel layout (output-split on 4 and 8
# waves, k-sliced, split-K, a GEMM that expands its own weight first).

GEMMS = (
    # (m, n, k, N, M, tile or None (planner), split)
    (333, 200, 1040, 2, 4, None, 1),
    (333, 200, 1040, 2, 8, 0, 1),        # compact weight, expanded inside the workgroups
    (333, 200, 1040, 1, 8, 6, 1),        # 8 waves
    (333, 200, 1040, 2, 4, 3, 2),        # split-K
    (100, 256, 256, 2, 4, None, 1),      # k-sliced
    (333, 200, 1040, 4, 8, 0, 1),        # mask layout: the dense kernel
    (2000, 512, 512, 8, 8, None, 1),     # dense weight
)


def _carry(m, n, k, N, M, tile, split, expand_self, job_N, job_M, seed):
    import torch
    rng = np.random.default_rng(seed)
    X = rng.integers(-128, 128, (m, k), dtype=np.int64).astype(np.int8)
    W = wl.random_nm(n, k, N, M, rng, full=True)
    ref = oracle.matmul_i8(X, W)
    Wj = wl.random_nm(96, 1024, job_N, job_M, rng, full=True)
    pj = nmspmm.compress(Wj, job_N, job_M)
    dj = nmspmm.DeviceWeight.from_packed(pj)
    e, nbytes = nmspmm.expand_size(pj.desc)
    want = torch.full((nbytes,), SENTINEL, dtype=torch.uint8, device="cuda")
    nmspmm.expand(dj, out=want)
    out = torch.full((nbytes + GUARD,), SENTINEL, dtype=torch.uint8, device="cuda")
    job, ew = nmspmm.expand_job(dj, out)
    Xd = torch.from_numpy(X).cuda()
    Y = torch.full((m, n), -7, dtype=torch.int32, device="cuda")
    dense = N == M
    if dense:
        plan = None if tile is None else nmspmm.make_plan(nmspmm.NM_KIND_DENSE, tile, split)
        nmspmm.gemm_i8_dense(Xd, torch.from_numpy(W).cuda(), Y=Y, plan=plan, job=job)
    else:
        p = nmspmm.compress(W, N, M)
        plan = None if tile is None else nmspmm.make_plan(p.desc.kind, tile, split, expand_self)
        nmspmm.spmm(Xd, nmspmm.DeviceWeight.from_packed(p), Y=Y, plan=plan, job=job)
    torch.cuda.synchronize()
    assert np.array_equal(Y.cpu().numpy(), ref)
    h = out.cpu().numpy()
    assert (h[nbytes:] == SENTINEL).all(), "write past the carried expansion"
    assert np.array_equal(h[:nbytes], want.cpu().numpy())
    return ew, Wj


@pytest.mark.parametrize("job_N,job_M", COMPACT)
@pytest.mark.parametrize("gemm", GEMMS)
def test_gemm_carries_an_expansion(gemm, job_N, job_M):
    m, n, k, N, M, tile, split = gemm
    _carry(m, n, k, N, M, tile, split, 0, job_N, job_M, seed=10 * GEMMS.index(gemm) + COMPACT.index((job_N, job_M)))


def test_gemm_that_expands_its_own_weight_carries_another():
    # the call launches the expansion of its own weight, then the GEMM with the carried one
    ew, Wj = _carry(2000, 256, 1024, 2, 8, 0, 1, 1, 4, 8, seed=3)
    # and the carried expansion is usable as a weight of its own
    import torch
    rng = np.random.default_rng(4)
    X = rng.integers(-128, 128, (150, 1024), dtype=np.int64).astype(np.int8)
    Y = torch.full((150, 96), -7, dtype=torch.int32, device="cuda")
    nmspmm.spmm(torch.from_numpy(X).cuda(), ew, Y=Y)
    torch.cuda.synchronize()
    assert np.array_equal(Y.cpu().numpy(), oracle.matmul_i8(X, Wj))


def test_no_tokens_still_runs_the_job():
    import torch
    rng = np.random.default_rng(8)
    Wj = wl.random_nm(64, 256, 1, 4, rng, full=True)
    pj = nmspmm.compress(Wj, 1, 4)
    dj = nmspmm.DeviceWeight.from_packed(pj)
    _, nbytes = nmspmm.expand_size(pj.desc)
    want = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    nmspmm.expand(dj, out=want)
    out = torch.full((nbytes,), SENTINEL, dtype=torch.uint8, device="cuda")
    job, _ = nmspmm.expand_job(dj, out)
    X = torch.empty((0, 128), dtype=torch.int8, device="cuda")
    W = torch.zeros((64, 128), dtype=torch.int8, device="cuda")
    nmspmm.gemm_i8_dense(X, W, Y=torch.empty((0, 64), dtype=torch.int32, device="cuda"), job=job)
    torch.cuda.synchronize()
    assert torch.equal(out, want)


def test_bad_job_launches_nothing():
    import ctypes
    import torch
    rng = np.random.default_rng(9)
    W = wl.random_nm(64, 256, 2, 4, rng, full=True)
    p = nmspmm.compress(W, 2, 4)
    dw = nmspmm.DeviceWeight.from_packed(p)
    Wj = wl.random_nm(64, 256, 2, 8, rng, full=True)
    pj = nmspmm.compress(Wj, 2, 8)
    dj = nmspmm.DeviceWeight.from_packed(pj)
    _, nbytes = nmspmm.expand_size(pj.desc)
    out = torch.full((nbytes,), SENTINEL, dtype=torch.uint8, device="cuda")
    X = torch.ones((100, 256), dtype=torch.int8, device="cuda")
    Y = torch.full((100, 64), -7, dtype=torch.int32, device="cuda")
    small = nmspmm.NmExpandJob(ctypes.pointer(pj.desc), dj.vals.data_ptr(), dj.meta.data_ptr(), out.data_ptr(),
                               nbytes - 16)
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.spmm(X, dw, Y=Y, job=small)
    assert e.value.status == nmspmm.NM_ERR_WORKSPACE
    stored = nmspmm.NmExpandJob(ctypes.pointer(p.desc), dw.vals.data_ptr(), dw.meta.data_ptr(), out.data_ptr(),
                                nbytes)
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.spmm(X, dw, Y=Y, job=stored)
    assert e.value.status == nmspmm.NM_ERR_ARG
    torch.cuda.synchronize()
    assert (Y == -7).all().item() and (out == SENTINEL).all().item()


def test_job_overlapping_the_gemm_is_refused():
    import ctypes
    import torch
    rng = np.random.default_rng(10)
    W = wl.random_nm(64, 256, 2, 4, rng, full=True)
    dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4))
    pj = nmspmm.compress(wl.random_nm(64, 256, 2, 8, rng, full=True), 2, 8)
    dj = nmspmm.DeviceWeight.from_packed(pj)
    _, nbytes = nmspmm.expand_size(pj.desc)
    X = torch.ones((100, 256), dtype=torch.int8, device="cuda")
    Y = torch.full((100, 64), -7, dtype=torch.int32, device="cuda")     # 25600 bytes >= nbytes
    assert Y.numel() * 4 >= nbytes
    for target in (Y, X):
        job = nmspmm.NmExpandJob(ctypes.pointer(pj.desc), dj.vals.data_ptr(), dj.meta.data_ptr(), target.data_ptr(),
                                 nbytes)
        with pytest.raises(nmspmm.NmError) as e:
            nmspmm.spmm(X, dw, Y=Y, job=job)
        assert e.value.status == nmspmm.NM_ERR_ARG
    torch.cuda.synchronize()
    assert (Y == -7).all().item() and (X == 1).all().item()
