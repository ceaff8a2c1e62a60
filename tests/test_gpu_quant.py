"""GPU parity of the INT8 chaining steps (through the C ABI) against the oracle.

* nm_quantize_f16 on every binary16 bit pattern (and a ragged tail), and on a
  large random activation tensor;
* the requantisation epilogue (int8 output of nm_spmm_out / nm_gemm_i8_dense_out)
  alone and together with the int32 and fp16 outputs, in every kernel layout
  and with split-K;
* two sparse linears chained through the int8 epilogue.

Codes are integers, so parity is bit-exact; the oracle decides them in binary32
as the kernels do.
"""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl
import gpu_util as gu

pytestmark = pytest.mark.gpu

I8_SENTINEL = -128   # q8 never produces -128


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = gu.torch()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    nmspmm.lib()
    yield
    torch.cuda.synchronize()


def i8_buffer(count):
    t = gu.torch()
    return t.full((count + gu.GUARD,), I8_SENTINEL, dtype=t.int8, device="cuda")


def fetch_i8(buf, count):
    h = buf.cpu().numpy()
    assert (h[count:] == I8_SENTINEL).all(), "write past the end of the int8 output"
    assert not (h[:count] == I8_SENTINEL).any(), "unwritten int8 output"
    return h[:count]


@pytest.mark.parametrize("inv_scale", [1.0, 0.37, 128.0, 3.0e-3])
def test_quantize_every_half(inv_scale):
    t = gu.torch()
    bits = np.concatenate([np.arange(65536, dtype=np.uint16), np.array([0x3800, 0x3E00, 0x4100, 0xBE00, 0x7C00,
                                                                        0xFC00, 0x7E00], np.uint16)])
    xd = t.from_numpy(bits.view(np.int16).copy()).cuda()
    out = i8_buffer(bits.size)
    nmspmm.quantize_f16(xd, inv_scale, xq=out[: bits.size])
    t.cuda.synchronize()
    assert np.array_equal(fetch_i8(out, bits.size), oracle.quantize_f16(bits, inv_scale))


def test_quantize_large_random():
    t = gu.torch()
    rng = np.random.default_rng(3)
    count = 18464 * 1024 + 5
    x = (rng.standard_normal(count) * 40).astype(np.float16)
    xd = t.from_numpy(x.view(np.int16)).cuda()
    out = i8_buffer(count)
    nmspmm.quantize_f16(xd, 1 / 0.3, xq=out[:count])
    t.cuda.synchronize()
    assert np.array_equal(fetch_i8(out, count), oracle.quantize_f16(x.view(np.uint16), np.float32(1 / 0.3)))


def test_quantize_errors():
    t = gu.torch()
    x = t.zeros(64, dtype=t.int16, device="cuda")
    xq = t.zeros(64, dtype=t.int8, device="cuda")
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.quantize_f16(x[1:], 1.0, xq=xq[:63])
    assert e.value.status == nmspmm.NM_ERR_ARG
    nmspmm.quantize_f16(x[:0], 1.0, xq=xq[:0])   # count 0: no-op


def qscales(ref, rng):
    """Per-channel multipliers that saturate about a fifth of the codes; some
    channels get 0.5 exactly so that odd accumulators round at a tie."""
    p = np.percentile(np.abs(ref.astype(np.float64)), 80, axis=0)
    q = (127.0 / np.maximum(p, 1.0)).astype(np.float32)
    q[rng.integers(0, q.size, max(1, q.size // 8))] = 0.5
    return q


PLANS = [None, (0, 1), (7, 1), (6, 1), (4, 1), (3, 2), (10, 2)]


@pytest.mark.parametrize("kind", ["2:4", "4:8", "dense"])
@pytest.mark.parametrize("plan", PLANS)
def test_requant_epilogue(kind, plan):
    t = gu.torch()
    m, n, k = 333, 200, 384
    print(f"requant {kind} plan={plan} m={m} n={n} k={k}", flush=True)
    rng = np.random.default_rng(17)
    X = rng.integers(-127, 128, (m, k)).astype(np.int8)
    if kind == "dense":
        W = rng.integers(-127, 128, (n, k)).astype(np.int8)
        kid = nmspmm.NM_KIND_DENSE
    else:
        N, M = map(int, kind.split(":"))
        W = wl.random_nm(n, k, N, M, rng, full=True)
        packed = nmspmm.compress(W, N, M)
        kid = packed.desc.kind
    ref = oracle.matmul_i8(X, W)
    qs = qscales(ref, rng)
    scale = rng.uniform(1e-6, 1e-3, n).astype(np.float32)
    want_q = oracle.requant_i8(ref, qs)
    Xd = t.from_numpy(X).cuda()
    qd, sd = t.from_numpy(qs).cuda(), t.from_numpy(scale).cuda()
    pl = None if plan is None else nmspmm.make_plan(kid, plan[0], plan[1])
    for outputs in ("q", "all"):
        Yq = i8_buffer(m * n)
        Yb, Yhb = gu.device_outputs(m, n, want_i32=outputs == "all", want_f16=outputs == "all")
        args = dict(Y=gu.view2d(Yb, m, n), scale=sd if outputs == "all" else None, Yh=gu.view2d(Yhb, m, n),
                    Yq=Yq[: m * n].view(m, n), qscale=qd, plan=pl)
        try:
            if kind == "dense":
                nmspmm.gemm_i8_dense(Xd, t.from_numpy(W).cuda(), **args)
            else:
                nmspmm.spmm(Xd, nmspmm.DeviceWeight.from_packed(packed), **args)
        except nmspmm.NmError as e:
            if e.status == nmspmm.NM_ERR_SHAPE and plan is not None:
                pytest.skip("tile does not fit this shape")
            raise
        t.cuda.synchronize()
        assert np.array_equal(fetch_i8(Yq, m * n).reshape(m, n), want_q)
        if outputs == "all":
            assert np.array_equal(gu.fetch(Yb, m, n), ref)
            gu.assert_f16_close(gu.fetch(Yhb, m, n), oracle.dequant_f16(ref, scale))


def test_two_linears_chained_in_int8():
    t = gu.torch()
    rng = np.random.default_rng(23)
    m, k0, n1, n2 = 197, 192, 768, 192
    X = rng.integers(-127, 128, (m, k0)).astype(np.int8)
    W1 = wl.random_nm(n1, k0, 2, 4, rng, full=True)
    W2 = wl.random_nm(n2, n1, 1, 4, rng, full=True)
    ref1 = oracle.matmul_i8(X, W1)
    qs1 = qscales(ref1, rng)
    X2 = oracle.requant_i8(ref1, qs1)
    ref2 = oracle.matmul_i8(X2, W2)
    p1, p2 = nmspmm.compress(W1, 2, 4), nmspmm.compress(W2, 1, 4)
    Xq = t.empty((m, n1), dtype=t.int8, device="cuda")
    Y2 = t.empty((m, n2), dtype=t.int32, device="cuda")
    nmspmm.spmm(t.from_numpy(X).cuda(), nmspmm.DeviceWeight.from_packed(p1), Yq=Xq, qscale=t.from_numpy(qs1).cuda())
    nmspmm.spmm(Xq, nmspmm.DeviceWeight.from_packed(p2), Y=Y2)
    t.cuda.synchronize()
    assert np.array_equal(Xq.cpu().numpy(), X2)
    assert np.array_equal(Y2.cpu().numpy(), ref2)


def test_requant_argument_errors():
    t = gu.torch()
    rng = np.random.default_rng(1)
    W = wl.random_nm(32, 128, 2, 4, rng)
    dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4))
    X = t.zeros((8, 128), dtype=t.int8, device="cuda")
    Yq = t.zeros((8, 32), dtype=t.int8, device="cuda")
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.spmm(X, dw, Yq=Yq, qscale=None)        # int8 output without its multipliers
    assert e.value.status == nmspmm.NM_ERR_ARG
    q = t.ones(33, dtype=t.float32, device="cuda")
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.spmm(X, dw, Yq=Yq, qscale=q[1:])      # misaligned multipliers
    assert e.value.status == nmspmm.NM_ERR_ARG
