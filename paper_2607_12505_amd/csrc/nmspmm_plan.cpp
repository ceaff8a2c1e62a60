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

size_t workspace_bytes(int split_k, int tiles, int m, int n) {
    (void)tiles;
    if (split_k <= 1) return 0;
    return kCounterBytes + (size_t)split_k * (size_t)m * (size_t)n * 4;
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

nm_status complete_plan(int kind, int m, int n, int k_steps, nm_plan *p) {
    if (!p || p->kind != kind || p->tile < 0 || p->tile >= kNumTiles) return NM_ERR_ARG;
    bool ok_split = false;
    for (int s : kSplitSet) ok_split |= (p->split_k == s);
    if (!ok_split || p->split_k > (k_steps > 0 ? k_steps : 1)) return NM_ERR_ARG;
    const TileCfg &t = kTiles[p->tile];
    p->tile_n = t.tile_n();
    p->tile_m = t.tile_m();
    const int64_t tiles = ceil_div(n, p->tile_n) * ceil_div(m > 0 ? m : 1, p->tile_m);
    if (t.layout == kRowStat) {
        // a fixed grid of workgroups, each walking an equal share of the tiles
        if (p->split_k != 1) return NM_ERR_ARG;
        const RowStatLds L = rowstat_lds(kind, t, k_steps);
        if (L.total > kLdsPerCu) return NM_ERR_SHAPE;
        const int64_t per_cu = (int64_t)(kLdsPerCu / L.total);
        const int64_t slots = (int64_t)device_cu_count() * per_cu;
        p->grid = (int)(tiles < slots ? tiles : slots);
        return NM_OK;
    }
    const int64_t grid = tiles * p->split_k;
    if (grid > 0x7fffffff) return NM_ERR_SHAPE;
    if (p->split_k > 1 && tiles > kMaxSplitTiles) return NM_ERR_ARG;
    // split-K partial sums are addressed with 32-bit byte offsets
    if (p->split_k > 1 && (int64_t)p->split_k * (m > 0 ? m : 1) * n * 4 >= ((int64_t)1 << 31)) return NM_ERR_SHAPE;
    p->grid = (int)grid;
    return NM_OK;
}

// Tile indices used by the rules below (see kTiles).
constexpr int kT256x256 = 0, kT128x128 = 2, kT128x64 = 4, kT64x64 = 6, kT32x32ks = 10, kT128x128rs = 11;

static int64_t tiles_of(int t, int m, int n) {
    return ceil_div(n, kTiles[t].tile_n()) * ceil_div(m, kTiles[t].tile_m());
}

nm_status make_plan(int kind, int m, int n, int k_steps, int out_mode, nm_plan *plan) {
    if (!plan || m < 0 || n < 1 || k_steps < 1) return NM_ERR_ARG;
    if ((out_mode & (NM_OUT_I32 | NM_OUT_F16 | NM_OUT_I8)) == 0) return NM_ERR_ARG;
    const int64_t cus = device_cu_count();
    const int mm = m > 0 ? m : 1;
    // Operands twice as heavy per k-step: dense weights and two 4:2 streams.
    const bool heavy = kind != NM_KIND_SP42;
    int tile;
    if (mm <= 512) {
        // Few tokens: too few output tiles to occupy the GPU.  Split the
        // reduction over the waves of each workgroup (k-sliced tile, merged in
        // LDS) when k is long enough and the 32 x 32 tiles do not oversubscribe.
        tile = (k_steps >= 4 && tiles_of(kT32x32ks, mm, n) <= 2 * cus) ? kT32x32ks : kT64x64;
    } else if (tiles_of(kT128x128, mm, n) < cus) {
        // Medium: the largest tile that still gives every compute unit one.
        tile = tiles_of(kT128x64, mm, n) >= cus ? kT128x64 : kT64x64;
    } else if (n <= 384 && k_steps >= 3) {
        // Narrow outputs: small tiles keep more workgroups per output row.
        tile = kT64x64;
    } else if (tiles_of(kT256x256, mm, n) >= 4 * cus || (heavy && n >= 3072)) {
        // Very large outputs: keep X resident and stream the weight when the
        // token block fits in LDS (short k, one-stream weights); otherwise the
        // biggest tile, which halves the operand traffic per output.
        const bool rs_fits = rowstat_lds(kind, kTiles[kT128x128rs], k_steps).total <= kLdsPerCu;
        tile = (!heavy && k_steps <= 6 && rs_fits) ? kT128x128rs : kT256x256;
    } else {
        tile = kT128x128;
    }
    plan->kind = kind;
    plan->tile = tile;
    plan->split_k = 1;
    return complete_plan(kind, m, n, k_steps, plan);
}

}  // namespace nmspmm
