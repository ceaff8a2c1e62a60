"""nm_expand (the decode of a compact weight as a pass of its own, Sec. 4.2)
through the C ABI: the expanded buffer, read by the header's formulas, holds
exactly the weight that was packed; the GEMM on the expanded descriptor gives
the oracle's product bit for bit; nothing is written past the buffer, and an
undersized buffer is rejected before anything is written."""
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
