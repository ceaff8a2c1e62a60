"""Helpers of the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the oracle (element by element, or at sampled
positions for the full-size workloads)."""
import numpy as np

import oracle
from paper_2607_12505_amd import nmspmm

INT32_SENTINEL = np.int32(-(2 ** 31))   # unreachable: |Y| < 128 * 128 * k < 2^31
F16_SENTINEL = np.uint16(0x7E01)        # a NaN the kernels never produce
GUARD = 256                             # elements of guard band after each output


def torch():
    import torch as t
    return t


def device_outputs(m, n, want_i32=True, want_f16=False):
    """Output buffers prefilled with sentinels, each followed by a guard band."""
    t = torch()
    Yb = Yhb = None
    if want_i32:
        Yb = t.full((m * n + GUARD,), int(INT32_SENTINEL), dtype=t.int32, device="cuda")
    if want_f16:
        Yhb = t.full((m * n + GUARD,), int(F16_SENTINEL.view(np.int16)), dtype=t.int16, device="cuda")
    return Yb, Yhb


def view2d(buf, m, n):
    return None if buf is None else buf[: m * n].view(m, n)


def fetch(buf, m, n):
    """Host copy of the output and a check that the guard band is untouched."""
    if buf is None:
        return None
    h = buf.cpu().numpy()
    guard = h[m * n:]
    if h.dtype == np.int32:
        assert (guard == INT32_SENTINEL).all(), "write past the end of Y"
        return h[: m * n].reshape(m, n)
    h = h.view(np.uint16)
    assert (guard == F16_SENTINEL).all(), "write past the end of Yh"
    return h[: m * n].reshape(m, n)


def run_sparse(X, packed, scale=None, want_i32=True, want_f16=False, plan=None, dw=None):
    t = torch()
    m, n = X.shape[0], packed.desc.n
    if dw is None:
        dw = nmspmm.DeviceWeight.from_packed(packed)
    Xd = t.from_numpy(np.ascontiguousarray(X)).cuda()
    sd = t.from_numpy(scale).cuda() if scale is not None else None
    Yb, Yhb = device_outputs(m, n, want_i32, want_f16)
    nmspmm.spmm(Xd, dw, Y=view2d(Yb, m, n), scale=sd, Yh=view2d(Yhb, m, n), plan=plan)
    t.cuda.synchronize()
    return fetch(Yb, m, n), fetch(Yhb, m, n)


def run_dense(X, W, scale=None, want_i32=True, want_f16=False, plan=None):
    t = torch()
    m, n = X.shape[0], W.shape[0]
    Xd = t.from_numpy(np.ascontiguousarray(X)).cuda()
    Wd = t.from_numpy(np.ascontiguousarray(W)).cuda()
    sd = t.from_numpy(scale).cuda() if scale is not None else None
    Yb, Yhb = device_outputs(m, n, want_i32, want_f16)
    nmspmm.gemm_i8_dense(Xd, Wd, Y=view2d(Yb, m, n), scale=sd, Yh=view2d(Yhb, m, n), plan=plan)
    t.cuda.synchronize()
    return fetch(Yb, m, n), fetch(Yhb, m, n)


def assert_f16_close(got, want):
    """binary16 parity: |g - r| <= 1e-3 |r| or <= 2^-24 (one subnormal step);
    infinities must match exactly; no NaN (the sentinel included) may appear."""
    g = got.view(np.float16).astype(np.float64)
    r = want.view(np.float16).astype(np.float64)
    assert not np.isnan(g).any(), "unwritten or NaN fp16 output"
    inf = np.isinf(r)
    assert np.array_equal(g[inf], r[inf])
    err = np.abs(np.where(inf, 0.0, g) - np.where(inf, 0.0, r))
    ok = (err <= 1e-3 * np.abs(np.where(inf, 0.0, r))) | (err <= 2.0 ** -24)
    bad = np.flatnonzero(~ok)
    assert bad.size == 0, f"{bad.size} fp16 mismatches, first at {bad[:5]}: {g.ravel()[bad[:5]]} vs {r.ravel()[bad[:5]]}"


def sample_positions(m, n, count, rng):
    """Random (i, j) plus the first/last rows and columns (tile edges, ragged tails)."""
    rows = [rng.integers(0, m, count)]
    cols = [rng.integers(0, n, count)]
    for i in {0, m - 1}:
        c = np.arange(0, n, max(1, n // 64))
        rows.append(np.full(c.size, i))
        cols.append(c)
    for j in {0, n - 1}:
        r = np.arange(0, m, max(1, m // 64))
        rows.append(r)
        cols.append(np.full(r.size, j))
    return np.concatenate(rows), np.concatenate(cols)


def check_sampled(X, W, Y, rng, count=3000, scale=None, Yh=None):
    rows, cols = sample_positions(X.shape[0], W.shape[0], count, rng)
    want = oracle.matmul_i8_sampled(X, W, rows, cols)
    got = Y[rows, cols] if Y is not None else None
    if got is not None:
        assert not (Y == INT32_SENTINEL).any(), "unwritten int32 output"
        mism = np.flatnonzero(got != want)
        assert mism.size == 0, f"{mism.size} int32 mismatches at {list(zip(rows[mism[:5]], cols[mism[:5]]))}"
    if Yh is not None:
        # each sampled value dequantised with its own channel's scale
        wh = oracle.dequant_f16(want[None, :], scale[cols])[0]
        assert_f16_close(Yh[rows, cols], wh)
