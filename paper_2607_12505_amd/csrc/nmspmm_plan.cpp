// The adaptive-parallelism planner (host only).
//
// The paper's rule (Sec. 4.3): raise split-K until there are enough blocks to
// occupy every compute unit ("parallelism priority"), keep the splits aligned
// with the matrix instruction's k granularity and the reduction overhead
// predictable ("controlled reduction"), and fall back to less splitting when
// k is short.  On MI355X the measured sweep over every (tile, split_k) of the
// ViT/DeiT/Swin workloads shows that a split of the reduction across the
// four waves of one workgroup, merged in LDS, beats a split across
// workgroups merged through global memory at every shape tried, so the rules
// choose among output tiles and k-sliced tiles, by token count, output tile
// count and output width; split_k > 1 is available to explicit plans.
#include <hip/hip_runtime.h>

#include <mutex>

#include "nmspmm_internal.h"

namespace nmspmm {

static const int kSplitSet[] = {1, 2, 4, 8};

size_t split_workspace_bytes(int split_k, int m, int n) {
    if (split_k <= 1) return 0;
    return kCounterBytes + (size_t)split_k * (size_t)m * (size_t)n * 4;
}

// The expanded weight always starts past the counter block (also without
// split-K), so no plan ever writes over the counters another plan relies on.
size_t expand_offset(int split_k, int m, int n) {
    const size_t used = split_k > 1 ? split_workspace_bytes(split_k, m, n) : kCounterBytes;
    return (used + 255) & ~(size_t)255;
}

size_t workspace_bytes(const nm_plan &p, int m, int n) {
    if (!p.expand) return split_workspace_bytes(p.split_k, m, n);
    return expand_offset(p.split_k, m, n) + (size_t)p.expand_bytes;
}

int64_t expanded_bytes(int kind, int n, int k) {
    if (!kind_is_compact(kind)) return 0;
    const int64_t F = (n + kFragRows - 1) / kFragRows, S = (k + kKStep - 1) / kKStep;
    return kind_is_sp42(kind) ? F * S * (kVBlock + kMBlock) : (int64_t)n * k;
}

int device_cu_count() {
    static std::mutex mu;
    static int cached[64];
    static bool init = false;
    std::lock_guard<std::mutex> lock(mu);
    if (!init) {
        for (int &c : cached) c = 0;
        init = true;
    }
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return 256;
    }
    if (cached[dev] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
            (void)hipGetLastError();
            cus = 256;
        }
        cached[dev] = cus;
    }
    return cached[dev];
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

nm_status complete_plan(int kind, int m, int n, int k, nm_plan *p) {
    if (!p || p->kind != kind || p->tile < 0 || p->tile >= kNumTiles) return NM_ERR_ARG;
    if (p->expand != 0 && (p->expand != 1 || !kind_is_compact(kind))) return NM_ERR_ARG;
    const int k_steps = (k + kKStep - 1) / kKStep;
    p->reserved = 0;
    p->expand_bytes = p->expand ? expanded_bytes(kind, n, k) : 0;
    bool ok_split = false;
    for (int s : kSplitSet) ok_split |= (p->split_k == s);
    if (!ok_split || p->split_k > (k_steps > 0 ? k_steps : 1)) return NM_ERR_ARG;
    const TileCfg &t = kTiles[p->tile];
    p->tile_n = t.tile_n();
    p->tile_m = t.tile_m();
    const int64_t tiles = ceil_div(n, p->tile_n) * ceil_div(m > 0 ? m : 1, p->tile_m);
    const int64_t grid = tiles * p->split_k;
    if (grid > 0x7fffffff) return NM_ERR_SHAPE;
    if (p->split_k > 1 && tiles > kMaxSplitTiles) return NM_ERR_ARG;
    // split-K partial sums are addressed with 32-bit byte offsets
    if (p->split_k > 1 && (int64_t)p->split_k * (m > 0 ? m : 1) * n * 4 >= ((int64_t)1 << 31)) return NM_ERR_SHAPE;
    p->grid = (int)grid;
    return NM_OK;
}

// Rows of output tiles from which a compact weight is expanded once per call.
constexpr int64_t kExpandTileRows = 32;

// Tile indices used by the rules below (see kTiles).
constexpr int kT128x128r2 = 0, kT128x64r2 = 1, kT64x128r2 = 2, kT64x64r2 = 3, kT256x256w8 = 4;
constexpr int kT128x32r2 = 5, kT128x128w8 = 6;
constexpr int kT64x64ks = 7, kT32x64ks = 8, kT64x32ks = 9, kT32x32ks = 10, kT128x160r2 = 11;

static int64_t tiles_of(int t, int m, int n) {
    return ceil_div(n, kTiles[t].tile_n()) * ceil_div(m, kTiles[t].tile_m());
}

nm_status make_plan(int kind, int m, int n, int k, int out_mode, nm_plan *plan) {
    if (!plan || m < 0 || n < 1 || k < 1) return NM_ERR_ARG;
    const int k_steps = (k + kKStep - 1) / kKStep;
    if ((out_mode & (NM_OUT_I32 | NM_OUT_F16 | NM_OUT_I8)) == 0) return NM_ERR_ARG;
    const int64_t cus = device_cu_count();
    const int mm = m > 0 ? m : 1;
    // Operands twice as heavy per k-step in matrix work: the kinds that run the
    // dense instruction (dense weights, and the mask layouts expanded to a
    // dense tile).
    const bool heavy = !kind_is_sp42(kind);
    // Rules fitted to an exhaustive timing of every tile on the ViT, DeiT and
    // Swin shapes (the paper's Table 1 methodology): above a few hundred
    // tokens the two-slot rings win -- their smaller LDS footprint keeps three
    // or more workgroups per compute unit, so one workgroup's loads overlap
    // another's compute and stores.
    int tile;
    if (mm <= 512) {
        // Few tokens: too few output tiles to occupy the GPU.  Split the
        // reduction over the waves of each workgroup (k-sliced 32 x 32 tile,
        // merged in LDS) while those tiles give at most 2 workgroups per CU.
        // For the heavier operands past one workgroup per CU, twice the tokens
        // per tile halve the weight fill (64 tokens, unless that pads m by more
        // than 15 %: then 64 channels); with a single k-step, 64 x 64.
        // Otherwise 64 x 64 with a 2-slot ring.
        const int64_t t32 = tiles_of(kT32x32ks, mm, n);
        if (t32 > 2 * cus)
            // many 32 x 32 tiles (the wide outputs): the k-sliced 64 x 64 tile
            // while it still fits two per CU (DeiT-B fc1 at batch 1: 9.0 us
            // against 9.9 for 64 x 64 with a ring), else 64 x 64
            tile = tiles_of(kT64x64ks, mm, n) <= 2 * cus ? kT64x64ks : kT64x64r2;
        else if (!heavy || t32 <= cus)
            tile = kT32x32ks;
        else if (k_steps == 1)
            tile = kT64x64r2;
        else
            tile = ceil_div(mm, 64) * 64 * 100 <= (int64_t)mm * 115 ? kT32x64ks : kT64x32ks;
    } else if (!heavy && k_steps >= 16 && k_steps <= 24 && mm <= 4096 && tiles_of(kT32x32ks, mm, n) <= 8 * cus) {
        // A few thousand tokens with a long reduction: the k-sliced 32 x 32
        // tile (the reduction split over the waves) still has more
        // workgroups than the output tiles of any ring tile (DeiT-B fc2 at
        // batch 8, 24 k-steps, inside the workload steps: 16.7 us against
        // 19 or more for 64 x 64; back to back, 64 x 64 is faster).  At 32
        // k-steps (Swin-B stage 4 fc2) 64 x 64 wins back to back by a third
        // and no in-network timing says otherwise, so the rule stops at 24.
        tile = kT32x32ks;
    } else if (k_steps <= 2) {
        // Very short reductions: the output stream dominates; small tiles
        // give the most workgroups in flight.  With one k-step and one-stream
        // weights, 128 channels x 32 tokens: the same number of workgroups
        // as 64 x 64, with output rows twice as long.
        tile = (!heavy && k_steps == 1 && n >= 384) ? kT128x32r2 : kT64x64r2;
    } else if (k_steps == 3) {
        // Three k-steps (DeiT-S, k = 384): 128 x 32 for one-stream weights,
        // 128 ch x 64 tok for the heavier operands (DeiT-S batch 64 proj,
        // dense, inside the steps: 12.5 us against 13.8-14.1 for 64 x 64; qkv
        // and fc1 within 1-3 %).
        tile = heavy ? kT128x64r2 : kT128x32r2;
    } else if (tiles_of(kT128x128r2, mm, n) < 4 * cus) {
        // Medium: with long reductions (8 k-steps or more) the operand fill
        // per output decides, so 128 x 128 as long as every compute unit
        // still gets a tile and the last tiles do not leave most units with
        // one while a few run two (1.25 tiles per unit or more); otherwise
        // half-height tiles (narrower for the heavier operands): DeiT-S batch
        // 64 fc2 (297 tiles of 128 x 128) 2:4 17.3 us against 18.5-18.7,
        // Swin-B stage 4 fc1 (312 tiles) dense 13.8-14.5 against 14.9-15.6.
        // A heavier operand whose channels fit one 128-row tile keeps 128 x
        // 128, which reads X once (Swin-B stage 1 fc2, 128 channels, dense:
        // 22.4-23.6 us against 23.7-25.3 for 64 x 128).
        const int64_t t128 = tiles_of(kT128x128r2, mm, n);
        if ((k_steps >= 8 && 4 * t128 >= 5 * cus) || (heavy && n <= 128 && t128 >= cus)) {
            tile = kT128x128r2;
        } else if (!heavy && k_steps < 8 && tiles_of(kT64x64r2, mm, n) <= 6 * cus) {
            // short reductions: 64 x 64 while it gives at most 6 workgroups
            // per CU (DeiT-B qkv and fc1 at batch 8: 11.1 and 13.1 us against
            // 13.4 and 15.0 for 128 x 64)
            tile = kT64x64r2;
        } else {
            // the heavier operands take 64 ch x 128 tok, except with long
            // reductions (12 k-steps or more), where 128 ch x 64 tok won in
            // every sweep inside the steps (DeiT-S batch 64 fc2 dense 18.8-19.6
            // us against 20.2-21.3, Swin-B stage 3 fc2 dense 17.4-18.0
            // against 18.0-19.1)
            tile = heavy && k_steps < 12 ? kT64x128r2 : kT128x64r2;
            // 64 x 64 when those would leave compute units without a tile,
            // and for one-stream weights when they already give 4 or more
            // workgroups per compute unit
            if (tiles_of(tile, mm, n) < cus || (!heavy && tiles_of(tile, mm, n) >= 4 * cus)) tile = kT64x64r2;
        }
    } else if (heavy) {
        // Large outputs, heavier operands: 128 x 128 on 8 waves (4 along the
        // channels x 2 along the tokens, twice the waves of the 4-wave tile to
        // overlap operand reads, matrix work and stores), except on the widest
        // outputs with long reductions (4096 channels or more, 24 k-steps or
        // more), where the 256 x 256 tile on 8 waves halves the operand fill
        // per output (6-13 % faster at k = 4096, n 4096 and 8192, m 8192-25216,
        // dense and 4:8).  Timed inside the steps of the ViT-L and DeiT-B
        // workloads with the 16-row tile groups (cold operands), 128 x 128 on
        // 8 waves won every other large shape (ViT-L qkv dense 82.7 us against
        // 88.4 on 4 waves, fc1 103.5 against 110.5) or tied within 2 %, except
        // the narrow outputs (512-1024 channels) with 8 or more k-steps: 160
        // tokens per tile on 4 waves, which reuses each weight slice over more
        // tokens (ViT-L fc2 dense 93.1 us against 102.7, DeiT-B batch 128 fc2
        // dense 66.8 against 74.5).
        if (n >= 4096 && k_steps >= 24)
            tile = kT256x256w8;
        else if (n >= 512 && n <= 1024 && k_steps >= 8)
            tile = kT128x160r2;
        else
            tile = kT128x128w8;
    } else {
        // Large outputs, 4:2-operand weights, timed the same way: long
        // reductions (24 k-steps or more) the 4-wave 128 x 128 tile, whose
        // larger per-wave fragment grid needs fewer operand reads per product
        // (ViT-L fc2 2:4 78.6 us, DeiT-B b128 fc2 60-62); otherwise 128 x 128
        // on 8 waves (ViT-L qkv and fc1 2:4: 70.4 and 87.2 us against 87.1
        // and 104.1 on the 256 x 256 tile, which the 16-row groups no longer
        // favour).
        tile = k_steps >= 24 ? kT128x128r2 : kT128x128w8;
    }
    plan->kind = kind;
    plan->tile = tile;
    plan->split_k = 1;
    // A compact weight is expanded inside every workgroup, ahead of its use,
    // when few rows of output tiles share it; with many rows the expansion
    // repeated per row costs more than one expansion pass per call.  1:4,
    // whose expansion is a few byte permutes, stays inside the workgroups
    // unless the reduction is long (24 k-steps or more: ViT-L fc2 81.5 us
    // expanded once against 87.3) or the output wide (4096 channels or more:
    // ViT-L fc1 86.2 against 89.7), or on the 256 x 256 tile (whose 8 waves
    // then need fewer registers).  The k-sliced tiles load the compact bytes
    // like X and expand them in registers, which the separate pass (a second
    // launch) never beats at the token counts they serve (DeiT-B fc2 at
    // batch 8, 1:4: 13.0 us against 16.1).
    // 1:8, whose expansion is a byte spread and a permute, likewise stays
    // inside below 2048 channels and 24 k-steps (DeiT-B batch 128 proj:
    // 26.8 us against 30.0 expanded once; qkv and fc1, 2304 and 3072 wide,
    // gain 2-6 % from the pass).  The pass costs a few microseconds whatever
    // the size (a second launch that waits for the first), so it is taken
    // only for GEMMs of 2^33 multiply-adds or more: inside the steps of
    // DeiT-S (at most 7.4e9) and Swin-B (at most 6.6e9) the in-kernel
    // expansion won every 2:8 and 4:8 GEMM, by 10-25 % (e.g. Swin-B stage 3
    // fc1 2:8 19.5 us against 24.3); from DeiT-B batch 128 proj up (1.5e10)
    // the pass wins (proj 2:8 30.0 us against 34.9).
    const bool many_rows = ceil_div(mm, kTiles[tile].tile_m()) >= kExpandTileRows;
    const bool k_sliced = kTiles[tile].layout == kKSliced;
    const bool long_gemm = (int64_t)mm * n * k >= ((int64_t)1 << 33);
    // With the expansion carried by an earlier launch the pass costs no
    // launch of its own.  Timed inside the workload steps with the expansions
    // carried: the 4:2-operand or dense kernel on the expanded weight then
    // beats the in-kernel decode for 1:8, 2:8 and the mask layouts at every
    // token count, k-sliced tiles included (DeiT-B batch 8 qkv 2:8 11.3 us
    // against 13.1, Swin-B stage 4 proj 2:8 9.0 against 12.1, ViT-L fc1 4:8
    // 112 against 127), and for 1:4, whose decode is a few permutes, only
    // with many rows of output-split tiles (DeiT-B batch 1 fc2 1:4 8.7 us
    // in-kernel against 10.3).
    const bool carried = (out_mode & NM_PLAN_EXPAND_CARRIED) != 0;
    bool once = long_gemm;
    if (kind == NM_KIND_C14) once = once && (k_steps >= 24 || n >= 4096 || tile == kT256x256w8);
    if (kind == NM_KIND_C18) once = once && (k_steps >= 24 || n >= 2048 || tile == kT256x256w8);
    if (carried)
        plan->expand = kind_is_compact(kind) && (kind != NM_KIND_C14 || (many_rows && !k_sliced)) ? 1 : 0;
    else
        plan->expand = kind_is_compact(kind) && many_rows && !k_sliced && once ? 1 : 0;
    return complete_plan(kind, m, n, k, plan);
}

}  // namespace nmspmm
