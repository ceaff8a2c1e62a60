"""nm_spmm_noalloc (the entry point that allocates nothing) against
nm_spmm_out with a caller workspace, through the C ABI: two calls in a row,
the second with a smaller input, for split-K plans (which use the library's
static scratch) and the planner's own plan; int32 bit-exact, fp16 within the
dequantisation tolerance, int8 bit-exact; and the size limit of the scratch."""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl
import gpu_util as gu

pytestmark = pytest.mark.gpu


def _inputs(m, n, k, N, M, seed):
    rng = np.random.default_rng(seed)
    X = rng.integers(-128, 128, (m, k)).astype(np.int8)
    W = wl.random_nm(n, k, N, M, rng, full=True)
    scale = rng.uniform(1e-6, 1e-3, n).astype(np.float32)
    qscale = rng.uniform(1e-5, 1e-3, n).astype(np.float32)
    return X, W, scale, qscale


def _outputs(torch, m, n):
    return (torch.full((m, n), -7, dtype=torch.int32, device="cuda"),
            torch.full((m, n), 0x7E01, dtype=torch.int16, device="cuda"),
            torch.full((m, n), 99, dtype=torch.int8, device="cuda"))


# (plan as (tile, split_k, expand) or None for the planner's, pattern)
CASES = [((3, 2, 0), (2, 4)), ((10, 4, 0), (2, 4)), ((0, 8, 0), (1, 8)), ((7, 2, 0), (4, 8)), (None, (2, 4)),
         ((0, 2, 1), (2, 8)), ((3, 1, 1), (4, 8))]


@pytest.mark.parametrize("plan,pat", CASES)
def test_noalloc_matches_workspace_call(plan, pat):
    torch = gu.torch()
    N, M = pat
    first = (197, 768, 3072)
    second = (61, 768, 3072)     # same weight, fewer tokens
    X1, W, scale, qscale = _inputs(*first, N, M, seed=5)
    X2 = np.random.default_rng(6).integers(-128, 128, (second[0], second[2])).astype(np.int8)
    packed = nmspmm.compress(W, N, M)
    dw = nmspmm.DeviceWeight.from_packed(packed)
    kind = packed.desc.kind
    p = None if plan is None else nmspmm.make_plan(kind, *plan)
    sd, qd = torch.from_numpy(scale).cuda(), torch.from_numpy(qscale).cuda()
    for X in (X1, X2):
        m, n = X.shape[0], W.shape[0]
        print(f"noalloc plan={plan} {N}:{M} m={m}", flush=True)
        Xd = torch.from_numpy(X).cuda()
        Ya, Yha, Yqa = _outputs(torch, m, n)
        nmspmm.spmm_noalloc(Xd, dw, Y=Ya, scale=sd, Yh=Yha, Yq=Yqa, qscale=qd, plan=p)
        Yb, Yhb, Yqb = _outputs(torch, m, n)
        nmspmm.spmm(Xd, dw, Y=Yb, scale=sd, Yh=Yhb, Yq=Yqb, qscale=qd, plan=p)
        torch.cuda.synchronize()
        ref = oracle.matmul_i8(X, W)
        assert np.array_equal(Ya.cpu().numpy(), ref)
        assert np.array_equal(Ya.cpu().numpy(), Yb.cpu().numpy())
        gu.assert_f16_close(Yha.cpu().numpy().view(np.uint16), oracle.dequant_f16(ref, scale))
        assert np.array_equal(Yha.cpu().numpy(), Yhb.cpu().numpy())
        assert np.array_equal(Yqa.cpu().numpy(), oracle.requant_i8(ref, qscale))
        assert np.array_equal(Yqa.cpu().numpy(), Yqb.cpu().numpy())


def test_noalloc_rejects_plans_beyond_the_scratch():
    torch = gu.torch()
    m, n, k = 2048, 1024, 1024    # split 8: 8 * 2048 * 1024 * 4 B = 64 MiB of partials > 32 MiB
    X, W, _, _ = _inputs(m, n, k, 2, 4, seed=7)
    dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4))
    plan = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 3, 8)
    assert nmspmm.workspace_size(plan, m, n) > nmspmm.NM_NOALLOC_SCRATCH_BYTES
    Y = torch.full((m, n), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.spmm_noalloc(torch.from_numpy(X).cuda(), dw, Y=Y, plan=plan)
    assert e.value.status == nmspmm.NM_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (Y.cpu().numpy() == -7).all()
