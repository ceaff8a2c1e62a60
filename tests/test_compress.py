"""Host packing (nm_compress / nm_decompress) against the N:M rule, the
documented physical layouts, hand-worked bytes and the oracle's canonical
packed form (CPU only)."""
import os

import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl

PATTERNS = [(1, 4), (2, 4), (3, 4), (4, 4)] + [(n, 8) for n in range(1, 9)]
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "nm_pack_layout_examples.txt")

# the layout the header assigns to each pattern
LAYOUT = {(1, 4): nmspmm.NM_LAYOUT_C14, (2, 4): nmspmm.NM_LAYOUT_SP42, (3, 4): nmspmm.NM_LAYOUT_DENSE,
          (4, 4): nmspmm.NM_LAYOUT_DENSE, (1, 8): nmspmm.NM_LAYOUT_C18, (2, 8): nmspmm.NM_LAYOUT_C28,
          (3, 8): nmspmm.NM_LAYOUT_MK3, (4, 8): nmspmm.NM_LAYOUT_MK4, (5, 8): nmspmm.NM_LAYOUT_MK5,
          (6, 8): nmspmm.NM_LAYOUT_DENSE, (7, 8): nmspmm.NM_LAYOUT_DENSE, (8, 8): nmspmm.NM_LAYOUT_DENSE}
# per-lane value and position bytes of the block layouts (header table)
LANE_BYTES = {nmspmm.NM_LAYOUT_SP42: (16, 4), nmspmm.NM_LAYOUT_C14: (8, 2), nmspmm.NM_LAYOUT_C18: (4, 2),
              nmspmm.NM_LAYOUT_C28: (8, 4), nmspmm.NM_LAYOUT_MK3: (12, 4), nmspmm.NM_LAYOUT_MK4: (16, 4),
              nmspmm.NM_LAYOUT_MK5: (20, 4)}
MASK_VALUES = {nmspmm.NM_LAYOUT_MK3: 3, nmspmm.NM_LAYOUT_MK4: 4, nmspmm.NM_LAYOUT_MK5: 5}


def lanes(vals, meta, d):
    """Yield (row, c0, value bytes, position word) per lane of every block,
    reading the buffers exactly as the header documents them."""
    VB, MB = LANE_BYTES[d.layout]
    F, S = d.n_frags, d.k_steps
    v = vals.view(np.int8).reshape(F * S * 64, VB)
    m = meta.view(np.uint8).reshape(F * S * 64, MB).astype(np.int64)
    words = sum(m[:, i] << (8 * i) for i in range(MB))
    for f in range(F):
        for s in range(S):
            for L in range(64):
                o = (f * S + s) * 64 + L
                yield 16 * f + L % 16, 128 * s + 32 * (L // 16), v[o], int(words[o])


def slots_documented(vals, meta, d):
    """Per lane and window (or 4-group): the list of (position, value) slots
    the header formula assigns, in slot order."""
    out = []
    for row, c0, vb, word in lanes(vals, meta, d):
        if d.layout == nmspmm.NM_LAYOUT_SP42:
            for g in range(8):
                out.append((row, c0 + 4 * g, [((word >> (4 * g + 2 * t)) & 3, int(vb[2 * g + t])) for t in range(2)]))
        elif d.layout == nmspmm.NM_LAYOUT_C14:
            for g in range(8):
                out.append((row, c0 + 4 * g, [((word >> (2 * g)) & 3, int(vb[g]))]))
        elif d.layout == nmspmm.NM_LAYOUT_C18:
            assert word >> 12 == 0
            for w in range(4):
                out.append((row, c0 + 8 * w, [((word >> (3 * w)) & 7, int(vb[w]))]))
        elif d.layout == nmspmm.NM_LAYOUT_C28:
            assert word >> 24 == 0
            for w in range(4):
                out.append((row, c0 + 8 * w, [((word >> (6 * w + 3 * t)) & 7, int(vb[2 * w + t])) for t in range(2)]))
        else:
            n = MASK_VALUES[d.layout]
            for w in range(4):
                mask = (word >> (8 * w)) & 0xFF
                pos = [p for p in range(8) if (mask >> p) & 1]
                assert len(pos) <= n
                # values past the last set bit are zero
                assert all(int(vb[n * w + j]) == 0 for j in range(len(pos), n))
                out.append((row, c0 + 8 * w, [(p, int(vb[n * w + j])) for j, p in enumerate(pos)]))
    return out


def decode_documented(p):
    """W rebuilt from the packed buffers by the header's formulas (padded to
    whole fragments and k-steps)."""
    d = p.desc
    if d.layout == nmspmm.NM_LAYOUT_DENSE:
        return np.ascontiguousarray(p.vals).view(np.int8).reshape(d.n, d.k).copy()
    Wr = np.zeros((16 * d.n_frags, 128 * d.k_steps), np.int64)
    for row, base, slots in slots_documented(p.vals, p.meta, d):
        for pos, val in slots:
            if val != 0:
                assert Wr[row, base + pos] == 0, "two nonzeros at one position"
                Wr[row, base + pos] = val
    return Wr.astype(np.int8)


@pytest.mark.parametrize("N,M", PATTERNS)
def test_roundtrip(N, M):
    rng = np.random.default_rng(N * 10 + M)
    for (n, k) in ((16, 128), (36, 192), (20, 4 * M * 3 + 16 * M)):
        if k % M or k % 16:
            continue
        W = wl.random_nm(n, k, N, M, rng)
        p = nmspmm.compress(W, N, M)
        assert p.desc.n == n and p.desc.k == k and p.desc.layout == LAYOUT[(N, M)] == p.desc.kind
        assert np.array_equal(nmspmm.decompress(p), W)
        # canonical idempotence
        p2 = nmspmm.compress(nmspmm.decompress(p), N, M)
        assert np.array_equal(p2.vals, p.vals) and np.array_equal(p2.meta, p.meta)


@pytest.mark.parametrize("N,M", PATTERNS)
def test_layout_matches_header_and_oracle(N, M):
    rng = np.random.default_rng(7 + N * 10 + M)
    n, k = 40, 320
    W = wl.random_nm(n, k, N, M, rng, full=bool(N % 2))
    p = nmspmm.compress(W, N, M)
    Wr = decode_documented(p)
    assert np.array_equal(Wr[:n, :k], W)
    assert not Wr[n:].any() and not Wr[:, k:].any()
    if p.desc.layout in (nmspmm.NM_LAYOUT_DENSE,) or p.desc.layout in MASK_VALUES:
        return
    # slot layouts: inside every window (4-group for SP42 and C14) the slots are
    # the oracle's canonical packing of that window
    win = 4 if p.desc.layout in (nmspmm.NM_LAYOUT_SP42, nmspmm.NM_LAYOUT_C14) else 8
    slots = len(slots_documented(p.vals, p.meta, p.desc)[0][2])
    for row, base, sl in slots_documented(p.vals, p.meta, p.desc):
        if row >= n or base >= k:
            assert all(v == 0 for _, v in sl)
            continue
        ov, oo = oracle.pack_logical(W[row:row + 1, base:base + win], slots, win)
        assert [pos for pos, _ in sl] == list(oo.ravel()) and [v for _, v in sl] == list(ov.ravel())


@pytest.mark.parametrize("N,M", PATTERNS)
def test_sizes_are_compact(N, M):
    n, k = 768, 192
    d = nmspmm.compress_size(n, k, N, M)
    F, S = -(-n // 16), -(-k // 128)
    assert (d.n_frags, d.k_steps) == (F, S)
    if d.layout == nmspmm.NM_LAYOUT_DENSE:
        assert (d.vals_bytes, d.meta_bytes) == (n * k, 0)
        return
    VB, MB = LANE_BYTES[d.layout]
    assert (d.vals_bytes, d.meta_bytes) == (64 * F * S * VB, 64 * F * S * MB)
    # N / M of the (padded) weight in values; position bits per weight as documented
    padded = 16 * F * 128 * S
    assert d.vals_bytes * M == padded * N
    bits_per_weight = {nmspmm.NM_LAYOUT_SP42: 1.0, nmspmm.NM_LAYOUT_C14: 0.5, nmspmm.NM_LAYOUT_C18: 0.5,
                       nmspmm.NM_LAYOUT_C28: 1.0}.get(d.layout, 1.0)
    assert d.meta_bytes * 8 == padded * bits_per_weight


def _golden_examples():
    ex, cur = [], None
    for line in open(GOLDEN):
        t = line.split("#", 1)[0].split()
        if not t:
            continue
        if t[0] == "example":
            cur = {"name": t[1], "N": int(t[2]), "M": int(t[3]), "w": [], "v": [], "m": []}
        elif t[0] == "w":
            cur["w"].append(tuple(int(x) for x in t[1:]))
        elif t[0] == "v":
            cur["v"].append((int(t[1]), int(t[2])))
        elif t[0] == "m":
            cur["m"].append((int(t[1]), int(t[2], 16)))
        elif t[0] == "end":
            ex.append(cur)
    return ex


@pytest.mark.parametrize("ex", _golden_examples(), ids=lambda e: e["name"])
def test_hand_worked_layout_bytes(ex):
    W = np.zeros((16, 128), np.int8)
    for r, c, v in ex["w"]:
        W[r, c] = v
    p = nmspmm.compress(W, ex["N"], ex["M"])
    vals = p.vals.view(np.int8)
    for off, v in ex["v"]:
        assert int(vals[off]) == v, (ex["name"], "vals", off)
    for off, b in ex["m"]:
        assert int(p.meta[off]) == b, (ex["name"], "meta", off)
    assert np.array_equal(nmspmm.decompress(p), W)
    assert np.array_equal(decode_documented(p), W)


def test_sizes():
    d = nmspmm.compress_size(768, 192, 2, 4)
    assert (d.n_frags, d.k_steps, d.layout) == (48, 2, nmspmm.NM_LAYOUT_SP42)
    assert d.vals_bytes == 48 * 2 * 1024 and d.meta_bytes == 48 * 2 * 256
    d = nmspmm.compress_size(100, 384, 4, 8)
    assert (d.n_frags, d.k_steps, d.layout) == (7, 3, nmspmm.NM_LAYOUT_MK4)
    assert d.vals_bytes == 7 * 3 * 1024 and d.meta_bytes == 7 * 3 * 256


def test_error_codes():
    W = np.zeros((16, 128), np.int8)
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(W, 2, 5)
    assert e.value.status == nmspmm.NM_ERR_UNSUPPORTED
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(W, 0, 4)
    assert e.value.status == nmspmm.NM_ERR_UNSUPPORTED
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(np.zeros((16, 132), np.int8), 2, 8)   # k % M
    assert e.value.status == nmspmm.NM_ERR_SHAPE
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(np.zeros((16, 136), np.int8), 2, 4)   # k % 16
    assert e.value.status == nmspmm.NM_ERR_SHAPE
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(np.zeros((18, 128), np.int8), 2, 4)   # n % 4
    assert e.value.status == nmspmm.NM_ERR_SHAPE
    bad = np.zeros((16, 128), np.int8)
    bad[5, 8:11] = 1                                          # 3 nonzeros in window 2
    with pytest.raises(nmspmm.NmError) as e:
        nmspmm.compress(bad, 2, 4)
    assert e.value.status == nmspmm.NM_ERR_PATTERN
    assert (e.value.bad_row, e.value.bad_group) == (5, 2)


def _rejects(p, vals=None, meta=None):
    with pytest.raises(nmspmm.NmError):
        nmspmm.decompress(nmspmm.Packed(p.vals if vals is None else vals, p.meta if meta is None else meta, p.desc))


def test_decompress_rejects_non_canonical():
    # SP42: slot 1 of group 0 at the position of slot 0 (both values nonzero)
    W = wl.random_nm(16, 128, 2, 4, np.random.default_rng(1), full=True)
    p = nmspmm.compress(W, 2, 4)
    meta = p.meta.copy()
    word = meta[:4].view(np.uint32)
    first = int(word[0]) & 3
    word[0] = (int(word[0]) & ~0xC) | (first << 2)
    _rejects(p, meta=meta)
    # a nonzero in the padding rows (n is 16 here, so use a 20-row weight)
    W2 = wl.random_nm(20, 128, 2, 4, np.random.default_rng(2), full=True)
    p2 = nmspmm.compress(W2, 2, 4)
    v2 = p2.vals.copy()
    v2[1024 * 1 + 16 * 10] = 5   # block of fragment 1, lane 10 -> row 26 >= 20
    _rejects(p2, vals=v2)


@pytest.mark.parametrize("N,M", [(1, 4), (1, 8), (2, 8), (3, 8), (4, 8), (5, 8)])
def test_compact_layouts_reject_non_canonical(N, M):
    rng = np.random.default_rng(N * 3 + M)
    W = wl.random_nm(16, 128, N, M, rng, full=False)
    W[0, :8] = 0                                              # lane 0's first window (or two groups) empty
    p = nmspmm.compress(W, N, M)
    lay = p.desc.layout
    VB, MB = LANE_BYTES[lay]
    # a zero value whose position is not the canonical one
    meta = p.meta.copy()
    if lay in MASK_VALUES:
        meta[0] = 0x01                                        # mask bit set for a zero value
    elif lay == nmspmm.NM_LAYOUT_C28:
        meta[:4].view(np.uint32)[0] = (int(meta[:4].view(np.uint32)[0]) & ~0x3F) | (1 | (2 << 3))
    else:
        meta[0] = (int(meta[0]) & ~0x3) | 1                   # group / window 0: position 1, value 0
    _rejects(p, meta=meta)
    # unused high position bits set
    if lay == nmspmm.NM_LAYOUT_C18:
        meta = p.meta.copy()
        meta[1] |= 0x80
        _rejects(p, meta=meta)
    if lay == nmspmm.NM_LAYOUT_C28:
        meta = p.meta.copy()
        meta[3] |= 0x01
        _rejects(p, meta=meta)
    # a mask layout: a nonzero value past the window's set bits
    if lay in MASK_VALUES:
        vals = p.vals.copy()
        vals[VB - 1] = 3                                      # last value slot of window 3 of lane 0
        nz = bin(int(p.meta[3])).count("1")
        if nz < MASK_VALUES[lay]:
            _rejects(p, vals=vals)


def test_generated_config_weights_roundtrip():
    for cfg in (0, 1, 2, 4):
        for g in wl.workload(cfg).gemms[:6]:
            if g.m > 20000:
                continue
            _, W, _ = wl.inputs_for(cfg, g)
            p = nmspmm.compress(W, g.N, g.M)
            assert np.array_equal(nmspmm.decompress(p), W)
