"""Pins of the CPU oracle against things other than itself (CPU only).

* the plain product against NumPy's int64 matmul (a library special case),
  one-hot closed forms, linearity and brute-force Python loops;
* the packed form against hand-worked examples (tests/golden), the round trip,
  the canonical-form invariants and brute-force window counts;
* the binary16 rounding exhaustively against the format's own grid
  (every half value and every midpoint) and against NumPy's converter;
* the int8 quantiser and requantiser against hand-worked codes (ties, saturation,
  NaN, infinities) and against NumPy's IEEE binary32 arithmetic on every
  binary16 input.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "nm_pack_examples.txt")
PATTERNS = [(1, 4), (2, 4), (3, 4), (4, 4)] + [(n, 8) for n in range(1, 9)]


def np_ref(X, W):
    return X.astype(np.int64) @ W.astype(np.int64).T


# ---------------------------------------------------------------- plain product

@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (3, 5, 7), (17, 9, 64), (33, 65, 192), (64, 16, 256)])
def test_matmul_matches_numpy(m, n, k):
    rng = np.random.default_rng(m * 1000 + n * 10 + k)
    X = rng.integers(-128, 128, (m, k)).astype(np.int8)
    W = rng.integers(-128, 128, (n, k)).astype(np.int8)
    assert np.array_equal(oracle.matmul_i8(X, W), np_ref(X, W))


def test_matmul_thread_count_does_not_matter():
    rng = np.random.default_rng(5)
    X = rng.integers(-128, 128, (37, 96)).astype(np.int8)
    W = rng.integers(-128, 128, (11, 96)).astype(np.int8)
    ys = [oracle.matmul_i8(X, W, nthreads=t) for t in (1, 2, 3, 8, 64)]
    for y in ys[1:]:
        assert np.array_equal(y, ys[0])


def test_matmul_bruteforce_tiny():
    rng = np.random.default_rng(11)
    X = rng.integers(-128, 128, (3, 8)).astype(np.int8)
    W = rng.integers(-128, 128, (4, 8)).astype(np.int8)
    Y = oracle.matmul_i8(X, W)
    for i in range(3):
        for j in range(4):
            s = 0
            for t in range(8):
                s += int(X[i, t]) * int(W[j, t])
            assert Y[i, j] == s


def test_matmul_one_hot_closed_forms():
    rng = np.random.default_rng(3)
    k, n = 64, 24
    W = rng.integers(-128, 128, (n, k)).astype(np.int8)
    # rows of X equal to 127 * e_t pick column t of W, scaled by 127
    X = np.zeros((k, k), np.int8)
    for t in range(k):
        X[t, t] = 127
    Y = oracle.matmul_i8(X, W)
    assert np.array_equal(Y, 127 * W.T.astype(np.int32))
    # one nonzero weight w at (j, t): column j of Y is w * X[:, t]
    Xr = rng.integers(-128, 128, (10, k)).astype(np.int8)
    W1 = np.zeros((n, k), np.int8)
    W1[7, 13] = -5
    Y1 = oracle.matmul_i8(Xr, W1)
    expect = np.zeros((10, n), np.int64)
    expect[:, 7] = -5 * Xr[:, 13].astype(np.int64)
    assert np.array_equal(Y1, expect)


def test_matmul_zero_and_linearity():
    rng = np.random.default_rng(4)
    X = rng.integers(-60, 60, (9, 32)).astype(np.int8)
    X2 = rng.integers(-60, 60, (9, 32)).astype(np.int8)
    W = rng.integers(-128, 128, (5, 32)).astype(np.int8)
    assert not oracle.matmul_i8(X, np.zeros_like(W)).any()
    lhs = oracle.matmul_i8((X.astype(np.int16) + X2).astype(np.int8), W)
    assert np.array_equal(lhs, oracle.matmul_i8(X, W) + oracle.matmul_i8(X2, W))


def test_matmul_bound_and_overflow():
    # |Y| <= 128 * 128 * k; with k >= 2^31 / 2^14 the extreme product leaves int32
    k = (1 << 17) + 64
    X = np.full((1, k), -128, np.int8)
    W = np.full((1, k), -128, np.int8)
    with pytest.raises(oracle.OracleError):
        oracle.matmul_i8(X, W)
    # just inside the range is exact
    k2 = 4096
    Y = oracle.matmul_i8(np.full((1, k2), -128, np.int8), np.full((1, k2), -128, np.int8))
    assert Y[0, 0] == 128 * 128 * k2


def test_matmul_sampled_matches_full():
    rng = np.random.default_rng(9)
    X = rng.integers(-128, 128, (50, 40)).astype(np.int8)
    W = rng.integers(-128, 128, (30, 40)).astype(np.int8)
    rows = rng.integers(0, 50, 200)
    cols = rng.integers(0, 30, 200)
    full = np_ref(X, W)
    assert np.array_equal(oracle.matmul_i8_sampled(X, W, rows, cols), full[rows, cols])


# ---------------------------------------------------------------- N:M rule

@pytest.mark.parametrize("N,M", PATTERNS)
def test_nm_check_bruteforce(N, M):
    rng = np.random.default_rng(N * 10 + M)
    for trial in range(20):
        W = rng.integers(-2, 3, (6, 4 * M)).astype(np.int8)  # many zeros, random counts
        counts = (W.reshape(6, 4, M) != 0).sum(axis=2)
        ok, br, bg = oracle.nm_check(W, N, M)
        assert ok == bool((counts <= N).all())
        if not ok:
            first = np.argwhere(counts > N)[0]
            assert (br, bg) == (first[0], first[1])


def test_nm_check_generated_weights():
    rng = np.random.default_rng(0)
    for (N, M) in PATTERNS:
        W, _ = wl.gen_w(32, 64, N, M, rng)
        assert oracle.nm_check(W, N, M)[0]
        if N < M:
            # the generator keeps exactly the top-N magnitudes, so (barring rounding to 0)
            # windows are mostly full and never exceed N
            cnt = (W.reshape(32, 64 // M, M) != 0).sum(axis=2)
            assert cnt.max() <= N and cnt.mean() > N - 0.5


# ---------------------------------------------------------------- packed form

def _golden():
    out = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = [p.split() for p in line.split("|")]
            N, M = map(int, parts[0])
            W = np.array(list(map(int, parts[1])), np.int8)[None, :]
            vals = np.array(list(map(int, parts[2])), np.int8)
            offs = np.array(list(map(int, parts[3])), np.uint8)
            X = np.array(list(map(int, parts[4])), np.int8)[None, :]
            y = int(parts[5][0])
            out.append((N, M, W, vals, offs, X, y))
    return out


def test_golden_examples():
    ex = _golden()
    assert len(ex) >= 6
    for (N, M, W, vals, offs, X, y) in ex:
        v, o = oracle.pack_logical(W, N, M)
        assert np.array_equal(v.ravel(), vals), (N, M, W)
        assert np.array_equal(o.ravel(), offs), (N, M, W)
        assert np.array_equal(oracle.unpack_logical(v, o, W.shape[1], M), W)
        assert oracle.spmm_packed(X, v, o, W.shape[1], M)[0, 0] == y
        assert oracle.matmul_i8(X, W)[0, 0] == y


@pytest.mark.parametrize("N,M", PATTERNS)
def test_pack_roundtrip_and_invariants(N, M):
    rng = np.random.default_rng(100 + N * 10 + M)
    W = wl.random_nm(13, 6 * M, N, M, rng)
    vals, offs = oracle.pack_logical(W, N, M)
    assert np.array_equal(oracle.unpack_logical(vals, offs, W.shape[1], M), W)
    # canonical form: positions inside the window, strictly ascending; nonzeros first
    # in position order; padding values are zero
    assert (offs < M).all()
    assert (np.diff(offs.astype(int), axis=2) > 0).all()
    G = W.shape[1] // M
    Wg = W.reshape(13, G, M)
    for j in range(13):
        for g in range(G):
            nz = np.flatnonzero(Wg[j, g])
            pads = [p for p in range(M) if p not in nz][: N - len(nz)]
            assert list(offs[j, g]) == sorted(list(nz) + pads)
            for s in range(N):
                assert vals[j, g, s] == Wg[j, g, offs[j, g, s]]
    # idempotence: packing the unpacked form gives the same packed form
    v2, o2 = oracle.pack_logical(oracle.unpack_logical(vals, offs, W.shape[1], M), N, M)
    assert np.array_equal(v2, vals) and np.array_equal(o2, offs)


def test_pack_rejects_violation():
    W = np.array([[1, 2, 3, 0, 0, 0, 0, 0]], np.int8)
    with pytest.raises(oracle.OracleError):
        oracle.pack_logical(W, 2, 4)


@pytest.mark.parametrize("N,M", PATTERNS)
def test_spmm_packed_equals_plain_product(N, M):
    rng = np.random.default_rng(200 + N * 10 + M)
    k = 8 * M
    W = wl.random_nm(19, k, N, M, rng)
    X = rng.integers(-128, 128, (23, k)).astype(np.int8)
    vals, offs = oracle.pack_logical(W, N, M)
    Y = oracle.spmm_packed(X, vals, offs, k, M)
    assert np.array_equal(Y, np_ref(X, W))


def test_spmm_packed_bruteforce_tiny():
    rng = np.random.default_rng(7)
    N, M, k = 2, 4, 16
    W = wl.random_nm(3, k, N, M, rng)
    X = rng.integers(-128, 128, (2, k)).astype(np.int8)
    vals, offs = oracle.pack_logical(W, N, M)
    Y = oracle.spmm_packed(X, vals, offs, k, M)
    for i in range(2):
        for j in range(3):
            s = 0
            for t in range(k):
                if W[j, t] != 0:
                    s += int(X[i, t]) * int(W[j, t])
            assert Y[i, j] == s


# ---------------------------------------------------------------- binary16 rounding

def _all_finite_halves():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    h = bits.view(np.float16)
    fin = np.isfinite(h)
    return bits[fin], h[fin].astype(np.float64)


def test_f16_every_half_is_a_fixed_point():
    bits, vals = _all_finite_halves()
    got = oracle.f64_to_f16(vals)
    # -0.0 keeps its sign bit
    assert np.array_equal(got, bits)


def test_f16_midpoints_round_to_even():
    # consecutive non-negative halves a < b (bit patterns p, p+1): the midpoint
    # rounds to whichever has an even last bit; just above/below go up/down.
    p = np.arange(0, 0x7BFF, dtype=np.uint16)  # up to the largest finite below 65504
    a = p.view(np.float16).astype(np.float64)
    b = (p + 1).view(np.float16).astype(np.float64)
    mid = (a + b) / 2  # exact in double
    got = oracle.f64_to_f16(mid)
    expect = np.where(p % 2 == 0, p, p + 1).astype(np.uint16)
    assert np.array_equal(got, expect)
    up = np.nextafter(mid, np.inf)
    dn = np.nextafter(mid, -np.inf)
    assert np.array_equal(oracle.f64_to_f16(up), (p + 1).astype(np.uint16))
    assert np.array_equal(oracle.f64_to_f16(dn), p)
    # negative side mirrors
    assert np.array_equal(oracle.f64_to_f16(-mid), expect | np.uint16(0x8000))


def test_f16_special_values():
    f = lambda x: int(oracle.f64_to_f16([x])[0])
    assert f(65504.0) == 0x7BFF
    assert f(65519.999) == 0x7BFF
    assert f(65520.0) == 0x7C00           # halfway to 2^16 rounds to even -> overflow
    assert f(1e300) == 0x7C00 and f(-1e300) == 0xFC00
    assert f(float("inf")) == 0x7C00 and f(float("-inf")) == 0xFC00
    assert f(float("nan")) & 0x7C00 == 0x7C00 and f(float("nan")) & 0x3FF
    assert f(2.0 ** -24) == 1              # smallest subnormal
    assert f(2.0 ** -25) == 0              # halfway to zero: even
    assert f(1.5 * 2.0 ** -24) == 2        # 1.5 ulp -> 2 (even)
    assert f(2.0 ** -14) == 0x0400         # smallest normal
    assert f(1.0) == 0x3C00 and f(-2.0) == 0xC000
    assert f(0.0) == 0 and f(-0.0) == 0x8000


def test_f16_matches_numpy_on_random_doubles():
    rng = np.random.default_rng(17)
    x = np.concatenate([
        rng.standard_normal(200000) * 10.0 ** rng.integers(-9, 6, 200000),
        rng.uniform(-70000, 70000, 10000),
    ])
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.f64_to_f16(x), want)


# ---------------------------------------------------------------- dequantisation

def test_dequant_exact_cases():
    rng = np.random.default_rng(21)
    Y = rng.integers(-2048, 2049, (16, 8)).astype(np.int32)
    # scale 1: every integer of magnitude <= 2048 is a half
    h = oracle.dequant_f16(Y, np.ones(8, np.float32))
    assert np.array_equal(h.view(np.float16).astype(np.float64), Y.astype(np.float64))
    # power-of-two scales are exact while the result stays normal
    sc = (2.0 ** -np.arange(8)).astype(np.float32)
    h = oracle.dequant_f16(Y, sc)
    assert np.array_equal(h.view(np.float16).astype(np.float64), Y * sc.astype(np.float64))


def test_dequant_matches_numpy():
    rng = np.random.default_rng(22)
    Y = rng.integers(-(1 << 26), 1 << 26, (64, 33)).astype(np.int32)
    sc = (rng.uniform(1e-7, 1e-4, 33)).astype(np.float32)
    want = (Y.astype(np.float64) * sc.astype(np.float64)[None, :]).astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.dequant_f16(Y, sc), want)


# ---------------------------------------------------------------- int8 (re)quantisation

def np_q8(v32):
    """Reference codes from NumPy's IEEE binary32 values: nearest-even, clamp, NaN -> 0."""
    with np.errstate(invalid="ignore"):
        r = np.rint(v32)
    r = np.where(np.isnan(r), 0, np.clip(r, -127, 127))
    return r.astype(np.int8)


def test_f16_decode_every_pattern_matches_numpy():
    bits = np.arange(65536, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    got = oracle.f16_to_f32(bits)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))   # signed zeros too


@pytest.mark.parametrize("inv_scale", [1.0, 0.37, 128.0, 3.0e-3, 1.0e4])
def test_quantize_every_half_matches_numpy(inv_scale):
    bits = np.arange(65536, dtype=np.uint16)
    with np.errstate(invalid="ignore"):
        ref = np_q8(bits.view(np.float16).astype(np.float32) * np.float32(inv_scale))
    assert np.array_equal(oracle.quantize_f16(bits, inv_scale), ref)


def test_quantize_hand_worked_codes():
    vals = [0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, 127.4, 200.0, -300.0, np.inf, -np.inf, np.nan, 0.0, -0.0, 3.25]
    want = [0, 2, 2, 0, -2, -2, 126, 127, 127, -127, 127, -127, 0, 0, 0, 3]
    bits = np.array(vals, np.float16).view(np.uint16)
    assert oracle.quantize_f16(bits, 1.0).tolist() == want
    # the multiplier is applied before rounding: 3 * 0.5 = 1.5 -> 2, 5 * 0.5 = 2.5 -> 2
    assert oracle.quantize_f16(np.array([3.0, 5.0, -7.0], np.float16).view(np.uint16), 0.5).tolist() == [2, 2, -4]


def test_requant_hand_worked_codes():
    Y = np.array([[0, 1, -1, 127, -127, 128, -128, 100000],
                  [3, 5, -3, -5, 7, 254, 255, -2 ** 31]], np.int32)
    got_1 = oracle.requant_i8(Y, np.ones(8, np.float32))
    assert got_1.tolist() == [[0, 1, -1, 127, -127, 127, -127, 127], [3, 5, -3, -5, 7, 127, 127, -127]]
    half = np.full(8, 0.5, np.float32)
    assert oracle.requant_i8(Y, half)[1].tolist() == [2, 2, -2, -2, 4, 127, 127, -127]
    per_ch = np.array([1, 1, 1, 0.5, 0.5, 0.25, 0.25, 1e-6], np.float32)
    assert oracle.requant_i8(Y, per_ch)[0].tolist() == [0, 1, -1, 64, -64, 32, -32, 0]


def test_requant_matches_numpy():
    rng = np.random.default_rng(11)
    Y = rng.integers(-2 ** 31, 2 ** 31, (37, 64), dtype=np.int64).astype(np.int32)
    Y[:, :16] = rng.integers(-40000, 40000, (37, 16))
    Y[:, 16:20] = rng.integers(2 ** 24 - 8, 2 ** 24 + 8, (37, 4))      # int -> binary32 rounding region
    q = np.exp(rng.uniform(np.log(1e-9), np.log(1e-2), 64)).astype(np.float32)
    q[:4] = np.float32(2.0 ** -22)
    ref = np_q8(Y.astype(np.float32) * q[None, :])
    assert np.array_equal(oracle.requant_i8(Y, q), ref)
