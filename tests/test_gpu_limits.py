"""The largest shapes the C ABI accepts, through the planner's own launch:
outputs of just under 2^29 elements and X of just under 2^32 bytes (the
kernels address outputs, X and the weight with 32-bit offsets).  Every output
is prefilled with a sentinel and followed by a guard band; the oracle checks
random positions, the first and last rows, and the last rows in full."""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl

pytestmark = pytest.mark.gpu

SENT = -(2 ** 31)
GUARD = 4096


def _device_x(torch, m, k, seed):
    """Seeded uniform int8 X [m x k] generated on the device in row chunks."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    X = torch.empty((m, k), dtype=torch.int8, device="cuda")
    step = max(1, (1 << 28) // k)
    for r in range(0, m, step):
        X[r:r + step].random_(-128, 128, generator=g)
    return X


def _check(torch, X, W, Ybuf, m, n, rng):
    Y = Ybuf[:m * n].view(m, n)
    torch.cuda.synchronize()
    assert (Ybuf[m * n:] == SENT).all().item(), "write past the end of Y"
    assert not (Y == SENT).any().item(), "unwritten output"
    rows = np.concatenate([rng.integers(0, m, 4000), np.zeros(64, np.int64), np.full(64, m - 1)])
    cols = np.concatenate([rng.integers(0, n, 4000), np.arange(64) % n, (n - 1 - np.arange(64)) % n])
    uniq, local = np.unique(rows, return_inverse=True)
    Xs = X[torch.from_numpy(uniq).cuda()].cpu().numpy()
    want = oracle.matmul_i8_sampled(Xs, W, local, cols)
    got = Y[torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()].cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches, first at {list(zip(rows[bad[:5]], cols[bad[:5]]))}"
    # the last rows (largest offsets) in full
    tail = 96
    Xt = X[m - tail:].cpu().numpy()
    assert np.array_equal(Y[m - tail:].cpu().numpy(), oracle.matmul_i8(Xt, W))


@pytest.mark.parametrize("sparse", [True, False])
def test_largest_output(sparse):
    import torch
    m, n, k = (1 << 20) - 16, 512, 128            # m n = 2^29 - 8192
    assert m * n < (1 << 29)
    rng = np.random.default_rng(11)
    X = _device_x(torch, m, k, 1234)
    W = wl.random_nm(n, k, 2, 4, rng, full=True) if sparse else rng.integers(-128, 128, (n, k)).astype(np.int8)
    Ybuf = torch.full((m * n + GUARD,), SENT, dtype=torch.int32, device="cuda")
    Y = Ybuf[:m * n].view(m, n)
    print(f"largest output: m={m} n={n} k={k} sparse={sparse}", flush=True)
    if sparse:
        nmspmm.spmm(X, nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4)), Y=Y)
    else:
        nmspmm.gemm_i8_dense(X, torch.from_numpy(W).cuda(), Y=Y)
    _check(torch, X, W, Ybuf, m, n, rng)
    del Ybuf, Y, X
    torch.cuda.empty_cache()


@pytest.mark.parametrize("sparse", [True, False])
def test_largest_input(sparse):
    import torch
    m, n, k = (1 << 22) - 64, 64, 1024           # m k = 2^32 - 65536 bytes of X
    assert m * k < (1 << 32) and m * n < (1 << 29)
    rng = np.random.default_rng(12)
    X = _device_x(torch, m, k, 4321)
    W = wl.random_nm(n, k, 1, 8, rng, full=True) if sparse else rng.integers(-128, 128, (n, k)).astype(np.int8)
    Ybuf = torch.full((m * n + GUARD,), SENT, dtype=torch.int32, device="cuda")
    Y = Ybuf[:m * n].view(m, n)
    print(f"largest input: m={m} n={n} k={k} sparse={sparse}", flush=True)
    if sparse:
        nmspmm.spmm(X, nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 1, 8)), Y=Y)
    else:
        nmspmm.gemm_i8_dense(X, torch.from_numpy(W).cuda(), Y=Y)
    _check(torch, X, W, Ybuf, m, n, rng)
    del Ybuf, Y, X
    torch.cuda.empty_cache()


def test_one_past_the_limits_is_refused():
    import torch
    X = torch.zeros((1 << 20, 16), dtype=torch.int8, device="cuda")
    W = torch.zeros((512, 16), dtype=torch.int8, device="cuda")
    Y = torch.empty((1 << 20, 512), dtype=torch.int32, device="cuda")      # m n = 2^29
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.gemm_i8_dense(X, W, Y=Y)
    assert e.value.status == nmspmm.NM_ERR_SHAPE
