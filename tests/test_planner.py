"""Adaptive-parallelism planner (paper Sec. 4.3) on the host (CPU only;
without a GPU the library assumes 256 compute units)."""
import itertools

import pytest

from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl

CUS = 256


def all_shapes():
    seen = set()
    for cfg in range(5):
        for g in wl.workload(cfg).gemms:
            key = (g.m, g.k, g.n, g.N, g.M)
            if key not in seen:
                seen.add(key)
                yield key
    for m, n, k in itertools.product((1, 17, 64, 197, 512), (128, 1024), (128, 1024)):
        yield (m, k, n, 2, 4)


@pytest.mark.parametrize("shape", list(all_shapes()))
def test_plan_rules(shape):
    m, k, n, N, M = shape
    d = nmspmm.compress_size(n, k, N, M)
    for out in (nmspmm.NM_OUT_I32, nmspmm.NM_OUT_F16, nmspmm.NM_OUT_I32 | nmspmm.NM_OUT_F16):
        p = nmspmm.spmm_plan(d, m, out)
        assert p.kind == d.kind
        assert p.split_k in (1, 2, 4, 8)
        tn, tm = nmspmm.tile_info(p.tile)
        tiles = -(-n // tn) * -(-m // tm)
        assert p.grid == tiles * p.split_k
        # the reduction is split inside workgroups, never across them; a
        # compact weight shared by many rows of output tiles is expanded once
        # per call into the workspace, past the counter block
        assert p.split_k == 1
        rows = -(-m // tm)
        compact = d.layout not in (nmspmm.NM_LAYOUT_SP42, nmspmm.NM_LAYOUT_DENSE)
        long_k, on_256 = -(-k // 128) >= 24, (tn, tm) == (256, 256)
        once = {nmspmm.NM_KIND_C14: long_k or n >= 4096 or on_256,
                nmspmm.NM_KIND_C18: long_k or n >= 2048 or on_256}.get(d.kind, True) and m * n * k >= 2 ** 33
        k_sliced = "k_gemm_ks" in nmspmm.plan_kernel_name(p)
        assert p.expand == int(compact and rows >= 32 and not k_sliced and once)
        if p.expand:
            F, S = -(-n // 16), -(-k // 128)
            want = F * S * 1280 if d.kind in (nmspmm.NM_KIND_C14, nmspmm.NM_KIND_C18, nmspmm.NM_KIND_C28) else n * k
            assert p.expand_bytes == want
            assert nmspmm.workspace_size(p, m, n) == 16384 + want
        else:
            assert p.expand_bytes == 0 and nmspmm.workspace_size(p, m, n) == 0
        # with the expansion carried by an earlier launch, every compact weight
        # is expanded once per call (1:4 only with many rows of output-split
        # tiles); the tile and split stay the same
        c = nmspmm.spmm_plan(d, m, out | nmspmm.NM_PLAN_EXPAND_CARRIED)
        assert (c.tile, c.split_k, c.grid) == (p.tile, p.split_k, p.grid)
        assert c.expand == int(compact and (d.kind != nmspmm.NM_KIND_C14 or (rows >= 32 and not k_sliced)))
        # deterministic
        q = nmspmm.spmm_plan(d, m, out)
        assert q.as_dict() == p.as_dict()
        dp = nmspmm.dense_plan(m, n, k, out)
        assert dp.kind == nmspmm.NM_KIND_DENSE and dp.split_k == 1


def test_small_token_counts_split_the_reduction_inside_workgroups():
    # DeiT-Base fc2 at batch 1: 197 tokens x 768 channels, k = 3072 (24 k-steps):
    # 64 x 64 tiles would leave 208 of 256 compute units idle, so the planner
    # takes the k-sliced 32 x 32 tile (the four waves split the reduction)
    d = nmspmm.compress_size(768, 3072, 2, 4)
    p = nmspmm.spmm_plan(d, 197, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (32, 32) and p.split_k == 1 and p.grid >= 128
    # ... and with two k-steps too (DeiT-Tiny fc1, k = 192)
    d = nmspmm.compress_size(768, 192, 2, 4)
    p = nmspmm.spmm_plan(d, 197, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (32, 32)
    # but the k-sliced 64 x 64 tile when 32 x 32 tiles would oversubscribe
    # (DeiT-Base fc1 at batch 1), while it fits twice per compute unit
    d = nmspmm.compress_size(3072, 768, 2, 4)
    p = nmspmm.spmm_plan(d, 197, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (64, 64) and nmspmm.plan_kernel_name(p) == "k_gemm_ks<1, 4, 4, 3>"
    d = nmspmm.compress_size(8192, 768, 2, 4)       # ... and 64 x 64 with a ring beyond that
    p = nmspmm.spmm_plan(d, 512, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (64, 64) and nmspmm.plan_kernel_name(p) == "k_gemm<1, 2, 2, 2, 2, 2>"
    # a few thousand tokens with a long reduction: k-sliced 32 x 32 too
    # (DeiT-Base fc2 at batch 8), not for the heavier operands
    d = nmspmm.compress_size(768, 3072, 2, 4)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 1576, 1)) == "k_gemm_ks<1, 2, 2, 3>"
    assert "k_gemm_ks" not in nmspmm.plan_kernel_name(nmspmm.dense_plan(1576, 768, 3072, 1))
    # a single k-step splits too (the paper's grid at k = 128)
    d = nmspmm.compress_size(1024, 128, 2, 4)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 256, 1)) == "k_gemm_ks<1, 2, 2, 3>"
    # heavier operands past one 32 x 32 tile per CU: 64 tokens per tile ...
    p = nmspmm.dense_plan(512, 1024, 512, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (32, 64) and "k_gemm_ks" in nmspmm.plan_kernel_name(p)
    # ... or 64 channels when 64-token tiles would pad m by more than 15 % (197 -> 256)
    p = nmspmm.dense_plan(197, 2304, 768, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (64, 32) and "k_gemm_ks" in nmspmm.plan_kernel_name(p)
    # ... and 64 x 64 with a single k-step
    p = nmspmm.dense_plan(512, 1024, 128, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (64, 64) and "k_gemm<" in nmspmm.plan_kernel_name(p)


def test_large_shapes_use_large_tiles():
    d = nmspmm.compress_size(3072, 768, 2, 4)
    p = nmspmm.spmm_plan(d, 25216, nmspmm.NM_OUT_I32)    # DeiT-Base fc1 at batch 128
    assert nmspmm.plan_kernel_name(p) == "k_gemm<1, 4, 2, 2, 4, 2>"   # 128 x 128 on 8 waves, 2-slot ring
    d = nmspmm.compress_size(3072, 1024, 4, 8)
    p = nmspmm.spmm_plan(d, 18464, nmspmm.NM_OUT_I32)    # ViT-L qkv, 4:8 weight: expanded once, dense kernel
    assert (p.tile_n, p.tile_m) == (128, 128) and nmspmm.plan_kernel_name(p) == "k_gemm<3, 4, 2, 2, 4, 2>"
    assert p.expand == 1
    # 4:2-operand weights: 128 x 128 on 8 waves up to 23 k-steps (ViT-L qkv
    # and fc1); long reductions, the 4-wave 128 x 128 tile (DeiT-B fc2 at
    # batch 128)
    d = nmspmm.compress_size(4096, 1024, 2, 4)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 18464, 1)) == "k_gemm<1, 4, 2, 2, 4, 2>"
    d = nmspmm.compress_size(3072, 1024, 1, 4)         # 1:4 on 3072 channels: expanded inside the workgroups
    p = nmspmm.spmm_plan(d, 18464, 1)
    assert nmspmm.plan_kernel_name(p) == "k_gemm<2, 4, 2, 2, 4, 2>" and p.expand == 0
    d = nmspmm.compress_size(4096, 1024, 1, 4)         # ... on 4096 channels expanded once, 4:2 kernel
    p = nmspmm.spmm_plan(d, 18464, 1)
    assert nmspmm.plan_kernel_name(p) == "k_gemm<1, 4, 2, 2, 4, 2>" and p.expand == 1
    d = nmspmm.compress_size(1024, 4096, 1, 4)         # ... and with 32 k-steps too
    p = nmspmm.spmm_plan(d, 18464, 1)
    assert nmspmm.plan_kernel_name(p) == "k_gemm<1, 2, 2, 4, 4, 2>" and p.expand == 1
    p = nmspmm.spmm_plan(d, 197, 1)                     # ... expanded inside the workgroups at batch 1
    assert p.expand == 0 and nmspmm.plan_kernel_name(p).startswith("k_gemm_ks<2,")
    d = nmspmm.compress_size(768, 3072, 2, 4)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 25216, 1)) == "k_gemm<1, 2, 2, 4, 4, 2>"
    # the dense baseline of DeiT-B fc2 at batch 128 (768 channels, 24 k-steps):
    # 128 channels x 160 tokens on 4 waves, and the same for ViT-L fc2 and proj;
    # wider dense outputs keep 128 x 128 on 8 waves (DeiT-B qkv)
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(25216, 768, 3072, 1)) == "k_gemm<3, 2, 2, 4, 5, 2>"
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(18464, 1024, 4096, 1)) == "k_gemm<3, 2, 2, 4, 5, 2>"
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(18464, 1024, 1024, 1)) == "k_gemm<3, 2, 2, 4, 5, 2>"
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(25216, 2304, 768, 1)) == "k_gemm<3, 4, 2, 2, 4, 2>"
    d = nmspmm.compress_size(1024, 4096, 4, 8)           # ... 4:8 on ViT-L fc2 too, expanded once
    p = nmspmm.spmm_plan(d, 18464, 1)
    assert (p.tile_n, p.tile_m) == (128, 160) and p.expand == 1
    # the widest outputs of the heavier operands with long reductions: 256 x 256 on 8 waves
    d = nmspmm.compress_size(4096, 4096, 4, 8)
    p = nmspmm.spmm_plan(d, 18464, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (256, 256) and nmspmm.plan_kernel_name(p) == "k_gemm<3, 2, 4, 8, 4, 3>"
    p = nmspmm.dense_plan(18464, 8192, 3072, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (256, 256)
    # ... and 128 x 128 on 8 waves for shorter ones (ViT-L fc1, 4:8 and its dense baseline)
    d = nmspmm.compress_size(4096, 1024, 4, 8)
    p = nmspmm.spmm_plan(d, 18464, nmspmm.NM_OUT_I32)
    assert (p.tile_n, p.tile_m) == (128, 128) and nmspmm.plan_kernel_name(p) == "k_gemm<3, 4, 2, 2, 4, 2>"
    p = nmspmm.dense_plan(18464, 4096, 1024, nmspmm.NM_OUT_I32)
    assert nmspmm.plan_kernel_name(p) == "k_gemm<3, 4, 2, 2, 4, 2>"
    d = nmspmm.compress_size(4096, 1024, 2, 4)           # 4:2-operand weight: 128 x 128 too
    assert (nmspmm.spmm_plan(d, 18464, 1).tile_n, nmspmm.spmm_plan(d, 18464, 1).tile_m) == (128, 128)
    d = nmspmm.compress_size(768, 3072, 2, 4)
    p = nmspmm.spmm_plan(d, 25216, nmspmm.NM_OUT_I32)    # fc2 at batch 128
    assert (p.tile_n, p.tile_m) == (128, 128)
    # three k-steps (DeiT-Small, k = 384): 128 channels x 32 tokens for
    # 4:2-operand weights, 128 channels x 64 tokens for the dense-tile ones
    d = nmspmm.compress_size(1152, 384, 2, 4)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 12608, 1)) == "k_gemm<1, 2, 2, 4, 1, 2>"
    d = nmspmm.compress_size(1152, 384, 4, 8)
    # expanded inside the workgroups (a GEMM of 5.6e9 multiply-adds, too short for the extra pass)
    assert nmspmm.plan_kernel_name(nmspmm.spmm_plan(d, 12608, 1)) == "k_gemm<7, 2, 2, 4, 2, 2>"
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(12608, 384, 384, 1)) == "k_gemm<3, 2, 2, 4, 2, 2>"
    d = nmspmm.compress_size(384, 384, 2, 4)
    assert (nmspmm.spmm_plan(d, 12608, 1).tile_n, nmspmm.spmm_plan(d, 12608, 1).tile_m) == (128, 32)
    # medium token counts, short reductions: 64 x 64 while it gives at most 4
    # workgroups per CU (DeiT-B qkv at batch 8, k = 768), else half-height
    # tiles (DeiT-B fc1 at batch 8), narrower for the dense-tile weights
    d = nmspmm.compress_size(2304, 768, 2, 4)
    assert (nmspmm.spmm_plan(d, 1576, 1).tile_n, nmspmm.spmm_plan(d, 1576, 1).tile_m) == (64, 64)
    d = nmspmm.compress_size(3072, 768, 2, 4)
    assert (nmspmm.spmm_plan(d, 1576, 1).tile_n, nmspmm.spmm_plan(d, 1576, 1).tile_m) == (64, 64)
    d = nmspmm.compress_size(4608, 768, 2, 4)
    assert (nmspmm.spmm_plan(d, 1576, 1).tile_n, nmspmm.spmm_plan(d, 1576, 1).tile_m) == (128, 64)
    d = nmspmm.compress_size(2304, 768, 4, 8)
    assert (nmspmm.spmm_plan(d, 1576, 1).tile_n, nmspmm.spmm_plan(d, 1576, 1).tile_m) == (64, 128)
    # ... but 64 x 64 for one-stream weights once half-height tiles give 4 or
    # more workgroups per compute unit (Swin-B stage 3 qkv, k = 512: 1176)
    d = nmspmm.compress_size(1536, 512, 2, 4)
    assert (nmspmm.spmm_plan(d, 6272, 1).tile_n, nmspmm.spmm_plan(d, 6272, 1).tile_m) == (64, 64)
    d = nmspmm.compress_size(1536, 512, 4, 8)
    assert (nmspmm.spmm_plan(d, 6272, 1).tile_n, nmspmm.spmm_plan(d, 6272, 1).tile_m) == (64, 128)
    # ... but 128 x 128 for long reductions while every compute unit gets a
    # tile (Swin-B stage 2 fc2, k = 1024: 392 tiles), not when fewer (stage 3
    # fc2, k = 2048: 196 tiles)
    d = nmspmm.compress_size(256, 1024, 2, 4)
    assert (nmspmm.spmm_plan(d, 25088, 1).tile_n, nmspmm.spmm_plan(d, 25088, 1).tile_m) == (128, 128)
    d = nmspmm.compress_size(512, 2048, 2, 4)
    assert (nmspmm.spmm_plan(d, 6272, 1).tile_n, nmspmm.spmm_plan(d, 6272, 1).tile_m) == (128, 64)
    # ... and half-height tiles when 128 x 128 gives fewer than 1.25 tiles per
    # compute unit (DeiT-S batch 64 fc2, k = 1536: 297 tiles; Swin-B stage 4
    # fc1, k = 1024: 312 tiles), narrower for the dense-tile weights
    d = nmspmm.compress_size(384, 1536, 2, 4)
    assert (nmspmm.spmm_plan(d, 12608, 1).tile_n, nmspmm.spmm_plan(d, 12608, 1).tile_m) == (128, 64)
    p = nmspmm.dense_plan(1568, 3072, 1024, 1)
    assert (p.tile_n, p.tile_m) == (64, 128)
    # ... except with 12 or more k-steps (DeiT-S batch 64 fc2, Swin-B stage 3
    # fc2 of the dense baseline): 128 ch x 64 tok
    p = nmspmm.dense_plan(12608, 384, 1536, 1)
    assert (p.tile_n, p.tile_m) == (128, 64)
    p = nmspmm.dense_plan(6272, 512, 2048, 1)
    assert (p.tile_n, p.tile_m) == (128, 64)
    d = nmspmm.compress_size(3072, 1024, 2, 4)
    assert (nmspmm.spmm_plan(d, 1568, 1).tile_n, nmspmm.spmm_plan(d, 1568, 1).tile_m) == (128, 64)
    # a dense-tile weight whose channels fit one 128-row tile keeps 128 x 128
    # at short reductions (Swin-B stage 1 fc2: 128 channels, k = 512)
    p = nmspmm.dense_plan(100352, 128, 512, 1)
    assert (p.tile_n, p.tile_m, p.tile) == (128, 128, 0)
    # ... or 64 x 64 when half-height tiles would leave compute units idle
    # (Swin-B stage 4 fc2 of the dense baseline: 96 tiles of 64 x 128)
    assert nmspmm.plan_kernel_name(nmspmm.dense_plan(1568, 1024, 4096, 1)) == "k_gemm<3, 2, 2, 2, 2, 2>"
    # one or two k-steps: 64 x 64 tiles (Swin-B stage 2 qkv, k = 256), and
    # 128 x 32 for one k-step of one-stream weights at least 384 wide (Swin-B
    # stage 1 qkv, k = 128; its proj, 128 wide, stays at 64 x 64)
    d = nmspmm.compress_size(384, 128, 2, 4)
    assert (nmspmm.spmm_plan(d, 100352, 1).tile_n, nmspmm.spmm_plan(d, 100352, 1).tile_m) == (128, 32)
    d = nmspmm.compress_size(128, 128, 2, 4)
    assert (nmspmm.spmm_plan(d, 100352, 1).tile_n, nmspmm.spmm_plan(d, 100352, 1).tile_m) == (64, 64)
    assert nmspmm.dense_plan(100352, 384, 128, 1).tile_m == 64
    d = nmspmm.compress_size(768, 256, 2, 4)
    assert (nmspmm.spmm_plan(d, 25088, 1).tile_n, nmspmm.spmm_plan(d, 25088, 1).tile_m) == (64, 64)


def test_forced_plan_completion():
    d = nmspmm.compress_size(768, 1024, 1, 8)
    p = nmspmm.spmm_plan_complete(d, 5000, nmspmm.make_plan(nmspmm.NM_KIND_C18, 0, 2, expand=1))
    assert p.expand_bytes == 48 * 8 * 1280 and (p.tile_n, p.tile_m) == (128, 128)
    # expanded weight after the counters and the split-K partials, 256-aligned
    part = 16384 + 2 * 5000 * 768 * 4
    assert nmspmm.workspace_size(p, 5000, 768) == -(-part // 256) * 256 + 48 * 8 * 1280
    with pytest.raises(nmspmm.NmError):      # only compact kinds expand
        nmspmm.spmm_plan_complete(nmspmm.compress_size(768, 1024, 2, 4), 100,
                                  nmspmm.make_plan(nmspmm.NM_KIND_SP42, 0, 1, expand=1))
    with pytest.raises(nmspmm.NmError):      # the descriptor's kind
        nmspmm.spmm_plan_complete(d, 100, nmspmm.make_plan(nmspmm.NM_KIND_C14, 0, 1))
    with pytest.raises(nmspmm.NmError):      # expand is 0 or 1
        nmspmm.spmm_plan_complete(d, 100, nmspmm.make_plan(nmspmm.NM_KIND_C18, 0, 1, expand=2))
    dm = nmspmm.compress_size(768, 1024, 4, 8)
    p = nmspmm.spmm_plan_complete(dm, 100, nmspmm.make_plan(nmspmm.NM_KIND_MK4, 3, 1, expand=1))
    assert p.expand_bytes == 768 * 1024


def test_forced_plan_validation():
    d = nmspmm.compress_size(256, 256, 2, 4)
    ok = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 0, 2)
    assert nmspmm.workspace_size(ok, 100, 256) > 0
    with pytest.raises(nmspmm.NmError):
        nmspmm.workspace_size(nmspmm.make_plan(nmspmm.NM_KIND_SP42, 99, 1), 100, 256)
    with pytest.raises(nmspmm.NmError):
        nmspmm.spmm_plan(d, -1)


def test_split_k_tile_limit():
    # split-K plans keep one counter per output tile in a fixed 16 KB block
    p = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 5, 2)
    assert nmspmm.workspace_size(p, 64 * 64, 64 * 64) == 16384 + 2 * 64 * 64 * 64 * 64 * 4
    p1 = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 5, 1)
    assert nmspmm.workspace_size(p1, 64 * 64, 64 * 64) == 0
