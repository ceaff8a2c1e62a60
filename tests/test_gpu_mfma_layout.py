"""Pins, on the GPU, the operand and result maps of the two matrix
instructions that the packed weight layout and the GEMM kernels rely on (one
wave, one instruction, per-lane operands through nm_probe_mfma_layout):

* v_smfmac_i32_16x16x128_i8: lane L holds row L % 16 of A; its 16 value bytes
  are the 8 aligned 4-groups of dense k in [32 (L // 16), +32), two values per
  group, and nibble g of its position word holds the two 2-bit positions of
  group g (low pair: first value).  B: lane L holds column L % 16, bytes 0..15
  for k in [16 (L // 16), +16), bytes 16..31 for k in [64 + 16 (L // 16), +16).
* v_mfma_i32_16x16x64_i8: lane L holds row L % 16 of A and column L % 16 of B,
  16 bytes each, for k in [16 (L // 16), +16).
* D (both): lane L holds rows 4 (L // 16) + e, e = 0..3, of column L % 16.

The position pairs are drawn from what the packer emits: two distinct
positions, ascending, or descending with a zero second value (a pad)."""
import itertools

import numpy as np
import pytest

from paper_2607_12505_amd import nmprobe, nmspmm

pytestmark = pytest.mark.gpu


def words(byte_rows):
    """[64, nbytes] int8 -> [64 * nbytes / 4] int32 (little-endian lane words)."""
    return np.ascontiguousarray(byte_rows.astype(np.int8)).view(np.int32).reshape(-1)


def run(kind, a_bytes, b_bytes, pos_words=None):
    import torch
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    a, b = dev(words(a_bytes)), dev(words(b_bytes))
    pos = dev(pos_words.astype(np.int32)) if pos_words is not None else None
    d = torch.empty(256, dtype=torch.int32, device="cuda")
    nmprobe.probe_mfma_layout(kind, a, b, pos, d)
    torch.cuda.synchronize()
    return d.cpu().numpy().reshape(64, 4)


def result_of(D):
    """16 x 16 int32 product -> the per-lane accumulator words."""
    out = np.zeros((64, 4), np.int64)
    for L in range(64):
        for e in range(4):
            out[L, e] = D[4 * (L // 16) + e, L % 16]
    return out


def sparse_dense_a(vals, pos):
    """Lane-major 4:2 A operand (values [64, 16], positions [64, 8, 2]) -> dense 16 x 128."""
    A = np.zeros((16, 128), np.int64)
    for L in range(64):
        for g in range(8):
            for s in range(2):
                A[L % 16, 32 * (L // 16) + 4 * g + pos[L, g, s]] += vals[L, 2 * g + s]
    return A


def sparse_b(b_bytes):
    B = np.zeros((128, 16), np.int64)
    for L in range(64):
        for j in range(16):
            B[16 * (L // 16) + j, L % 16] = b_bytes[L, j]
            B[64 + 16 * (L // 16) + j, L % 16] = b_bytes[L, 16 + j]
    return B


def pos_words_of(pos):
    w = np.zeros(64, np.int64)
    for g in range(8):
        w |= (pos[:, g, 0] | (pos[:, g, 1] << 2)) << (4 * g)
    return (w & 0xFFFFFFFF).astype(np.uint32).view(np.int32)


def random_sparse_operands(rng):
    pairs = [p for p in itertools.permutations(range(4), 2)]
    pos = np.array([[pairs[rng.integers(len(pairs))] for _ in range(8)] for _ in range(64)], np.int64)
    vals = rng.integers(-128, 128, (64, 16))
    # a descending pair is a pad: its second value is zero, as the packer writes it
    for L in range(64):
        for g in range(8):
            if pos[L, g, 1] < pos[L, g, 0]:
                vals[L, 2 * g + 1] = 0
    return vals, pos


def test_smfmac_maps_random_operands():
    rng = np.random.default_rng(11)
    for _ in range(4):
        vals, pos = random_sparse_operands(rng)
        b_bytes = rng.integers(-128, 128, (64, 32))
        got = run(nmspmm.NM_KIND_SP42, vals, b_bytes, pos_words_of(pos))
        want = result_of(sparse_dense_a(vals, pos) @ sparse_b(b_bytes))
        np.testing.assert_array_equal(got, want)


def test_smfmac_one_hot():
    # one value of A (lane L, group g, slot s at position p) times one byte of B:
    # exactly one output, at row L % 16 and the column of the B lane, when the
    # two dense k indices meet
    rng = np.random.default_rng(12)
    for L, g, s, p in [(0, 0, 0, 0), (5, 3, 1, 3), (17, 7, 0, 2), (38, 2, 1, 1), (63, 5, 0, 3)]:
        vals = np.zeros((64, 16), np.int64)
        pos = np.tile(np.array([0, 1]), (64, 8, 1))
        pos[L, g] = (p, 3 if p != 3 else 2) if s == 0 else (0 if p != 0 else 1, p)
        if s == 1 and pos[L, g, 1] < pos[L, g, 0]:
            pos[L, g] = (pos[L, g, 1], pos[L, g, 0])
            s = 0
        vals[L, 2 * g + s] = 3
        k = 32 * (L // 16) + 4 * g + pos[L, g, s]
        col = int(rng.integers(16))
        b_bytes = np.zeros((64, 32), np.int64)
        bl = (k % 64) // 16 * 16 + col
        b_bytes[bl, (k % 16) + (16 if k >= 64 else 0)] = 5
        got = run(nmspmm.NM_KIND_SP42, vals, b_bytes, pos_words_of(pos))
        want = np.zeros((16, 16), np.int64)
        want[L % 16, col] = 15
        np.testing.assert_array_equal(got, result_of(want))


def test_dense_mfma_maps_random_operands():
    rng = np.random.default_rng(13)
    for _ in range(4):
        a_bytes = rng.integers(-128, 128, (64, 16))
        b_bytes = rng.integers(-128, 128, (64, 16))
        A = np.zeros((16, 64), np.int64)
        B = np.zeros((64, 16), np.int64)
        for L in range(64):
            A[L % 16, 16 * (L // 16): 16 * (L // 16) + 16] = a_bytes[L]
            B[16 * (L // 16): 16 * (L // 16) + 16, L % 16] = b_bytes[L]
        got = run(nmspmm.NM_KIND_DENSE, a_bytes, b_bytes)
        np.testing.assert_array_equal(got, result_of(A @ B))


def test_extremes_do_not_saturate():
    # all -128 x -128 over the full k: 128 products of 16384 (smfmac: 64 of them
    # on stored values) stay exact in int32
    a_bytes = np.full((64, 16), -128)
    b_bytes = np.full((64, 16), -128)
    got = run(nmspmm.NM_KIND_DENSE, a_bytes, b_bytes)
    assert (got == 64 * 16384).all()
    pos = np.tile(np.array([0, 1]), (64, 8, 1))
    got = run(nmspmm.NM_KIND_SP42, np.full((64, 16), -128), np.full((64, 32), -128), pos_words_of(pos))
    assert (got == 64 * 16384).all()
