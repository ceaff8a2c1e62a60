"""GPU parity along every branch of the adaptive-parallelism planner (Sec.
4.3): one seeded shape per rule, for 2:4 (stored 4:2 operand), 1:4, 1:8 and
2:8 (compact, expanded to the 4:2 operand), 4:8 (mask layout expanded to a
dense tile) and dense weights, compared element by element with the oracle in the launch
configuration the planner picks (int32 and fp16 outputs, guard bands after
both).  The expected tile of each case documents the rule it exercises;
launches with 32 or more rows of tiles walk them in groups of 16 rows,
including a ragged last group, also with the reduction split across
workgroups."""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
import gpu_util as gu

pytestmark = pytest.mark.gpu

KS = "k_gemm_ks"
# (m, n, k, kind, expected (tile_n, tile_m), k-sliced?)
CASES = [
    (100, 256, 256, "sp", (32, 32), True),      # few tokens: k-sliced 32 x 32
    (100, 256, 128, "sp", (32, 32), True),      # ... also with a single k-step
    (512, 1024, 256, "dn", (32, 64), True),     # heavier operands past one tile per CU: 64 tokens
    (512, 1024, 256, "mk", (32, 64), True),
    (197, 2304, 256, "dn", (64, 32), True),     # ... or 64 channels when 64 tokens pad m too much
    (512, 1024, 128, "dn", (64, 64), False),    # ... and 64 x 64 with a single k-step
    (400, 4096, 128, "sp", (64, 64), True),     # more than 2 k-sliced 32 x 32 tiles per CU: k-sliced 64 x 64
    (512, 8192, 128, "sp", (64, 64), False),    # ... more than 2 of those too: 64 x 64 with a ring
    (3000, 512, 128, "sp", (128, 32), False),   # one k-step, one stream, >= 384 wide: 128 x 32
    (3000, 256, 128, "sp", (64, 64), False),    # ... narrower: 64 x 64
    (3000, 512, 256, "sp", (64, 64), False),    # two k-steps: 64 x 64
    (2000, 768, 384, "sp", (128, 32), False),   # three k-steps, one stream: 128 x 32
    (2000, 768, 384, "mk", (128, 64), False),   # ... heavier operands: 128 ch x 64 tok
    (5200, 1024, 1024, "sp", (128, 128), False),  # medium, long reduction: 128 x 128
    (4000, 1152, 1024, "sp", (128, 64), False),   # ... half-height under 1.25 such tiles per CU
    (1568, 3072, 1024, "dn", (64, 128), False),   # ... narrower for the heavier operands
    (33000, 128, 512, "dn", (128, 128), False),   # ... heavier operands 128 channels wide: 128 x 128
    (33000, 128, 512, "mk", (128, 128), False),
    (1600, 2304, 768, "sp", (64, 64), False),   # medium, short reduction: 64 x 64 up to 6 per CU
    (2560, 2560, 768, "sp", (128, 64), False),  # ... past that, half-height tiles
    (1600, 2304, 768, "dn", (64, 128), False),  # ... narrower for the heavier operands
    (6272, 512, 2048, "dn", (128, 64), False),  # ... but not with 12 or more k-steps
    (6272, 1536, 512, "sp", (64, 64), False),   # ... 64 x 64 past 4 half-height tiles per CU
    (8192, 2048, 512, "sp", (128, 128), False),  # large: 128 x 128
    (4096, 4096, 3072, "mk", (256, 256), False),  # large, heavier operands, 4096 wide, long reduction: 256 x 256
    (4096, 4096, 512, "mk", (128, 128), False),   # ... shorter reduction: 128 x 128 on 8 waves
    (16500, 1024, 1024, "dn", (128, 160), False),  # ... narrow outputs, 8+ k-steps: 160 tokens (ragged rows)
    (16500, 1024, 1024, "mk", (128, 160), False),  # ... the same for 4:8, expanded once
    # 32 or more rows of tiles: tiles walked in groups of 16 rows
    (8300, 3072, 2048, "sp", (128, 128), False),  # 65 tile rows: the last group has one row
    (5000, 1024, 512, "sp", (64, 64), False),     # 79 tile rows: the last group has 15
    (8192, 3072, 1024, "mk", (128, 128), False),
    (8192, 2048, 2048, "dn", (128, 128), False),
    # the compact kinds on the same rules
    (100, 256, 256, "c14", (32, 32), True),
    (100, 256, 256, "c18", (32, 32), True),
    (197, 2304, 256, "c28", (32, 32), True),
    (3000, 512, 128, "c18", (128, 32), False),
    (2000, 768, 384, "c28", (128, 32), False),
    (1600, 2304, 768, "c14", (64, 64), False),
    (2560, 2560, 768, "c14", (128, 64), False),
    (8192, 2048, 512, "c28", (128, 128), False),
    (8300, 3072, 2048, "c18", (128, 128), False),
]
PATTERN = {"sp": (2, 4), "mk": (4, 8), "c14": (1, 4), "c18": (1, 8), "c28": (2, 8)}


@pytest.mark.parametrize("m,n,k,kind,tile,ks", CASES)
def test_planner_branch_matches_oracle(m, n, k, kind, tile, ks):
    print(f"planner branch m={m} n={n} k={k} {kind}", flush=True)
    rng = np.random.default_rng(m * 31 + n * 7 + k)
    X = rng.integers(-128, 128, (m, k)).astype(np.int8)
    scale = rng.uniform(1e-6, 1e-3, n).astype(np.float32)
    if kind == "dn":
        W = rng.integers(-128, 128, (n, k)).astype(np.int8)
        plan = nmspmm.dense_plan(m, n, k, nmspmm.NM_OUT_I32 | nmspmm.NM_OUT_F16)
    else:
        from paper_2607_12505_amd import workloads as wl
        N, M = PATTERN[kind]
        W = wl.random_nm(n, k, N, M, rng, full=True)
        packed = nmspmm.compress(W, N, M)
        plan = nmspmm.spmm_plan(packed.desc, m, nmspmm.NM_OUT_I32 | nmspmm.NM_OUT_F16)
    name = nmspmm.plan_kernel_name(plan)
    assert (plan.tile_n, plan.tile_m) == tile and (KS in name) == ks, name
    if kind == "dn":
        Y, Yh = gu.run_dense(X, W, scale, want_i32=True, want_f16=True)
    else:
        Y, Yh = gu.run_sparse(X, packed, scale, want_i32=True, want_f16=True)
    ref = oracle.matmul_i8(X, W)
    assert np.array_equal(Y, ref), name
    gu.assert_f16_close(Yh, oracle.dequant_f16(ref, scale))


@pytest.mark.parametrize("split", [2, 4])
def test_grouped_order_with_split_k_matches_oracle(split):
    # 66 rows of 64 x 64 tiles, each split over the reduction: the grouped
    # order walks (row, split) pairs, 132 of them, the last group ragged
    m, n, k = 4200, 256, 1024
    print(f"grouped order split_k={split} m={m} n={n} k={k}", flush=True)
    rng = np.random.default_rng(4200 + split)
    X = rng.integers(-128, 128, (m, k)).astype(np.int8)
    from paper_2607_12505_amd import workloads as wl
    W = wl.random_nm(n, k, 2, 4, rng, full=True)
    packed = nmspmm.compress(W, 2, 4)
    plan = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 3, split)
    Y, _ = gu.run_sparse(X, packed, plan=plan)
    assert np.array_equal(Y, oracle.matmul_i8(X, W))
