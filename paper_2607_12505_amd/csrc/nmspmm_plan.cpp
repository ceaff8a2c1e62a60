// Tile table and the adaptive-parallelism planner (host only).
//
// The paper's rule (Sec. 4.3): raise split-K until there are enough blocks to
// occupy every compute unit ("parallelism priority"), take split-K from a
// small discrete set so that every split stays aligned with the matrix
// instruction's k granularity ("controlled reduction"), and fall back to a
// smaller split when k is short or the reduction would dominate.  Here the
// tile size is chosen first (largest tile that still fills the GPU with
// little padding waste), and split-K only when even the smallest tile leaves
// compute units idle.
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
    const int64_t grid = tiles * p->split_k;
    if (grid > 0x7fffffff) return NM_ERR_SHAPE;
    if (p->split_k > 1 && tiles > kMaxSplitTiles) return NM_ERR_ARG;
    p->grid = (int)grid;
    return NM_OK;
}

nm_status make_plan(int kind, int m, int n, int k_steps, int out_mode, nm_plan *plan) {
    if (!plan || m < 0 || n < 1 || k_steps < 1) return NM_ERR_ARG;
    if ((out_mode & (NM_OUT_I32 | NM_OUT_F16)) == 0) return NM_ERR_ARG;
    const int cus = device_cu_count();
    const int mm = m > 0 ? m : 1;
    // 1) the largest tile that gives at least one workgroup per compute unit
    //    while padding stays below 12.5 % of the useful outputs
    int best = -1;
    for (int i = 0; i < kNumTiles; ++i) {
        const TileCfg &t = kTiles[i];
        const int64_t tn = ceil_div(n, t.tile_n()), tm = ceil_div(mm, t.tile_m());
        const double waste = (double)(tn * t.tile_n()) * (double)(tm * t.tile_m()) / ((double)n * mm);
        if (tn * tm >= cus && waste <= 1.125) { best = i; break; }
    }
    int split = 1;
    if (best < 0) {
        // 2) otherwise the tile with the most workgroups (least padding on ties) ...
        int64_t most = -1;
        double most_waste = 0;
        for (int i = 0; i < kNumTiles; ++i) {
            const TileCfg &t = kTiles[i];
            const int64_t tn = ceil_div(n, t.tile_n()), tm = ceil_div(mm, t.tile_m());
            const double waste = (double)(tn * t.tile_n()) * (double)(tm * t.tile_m()) / ((double)n * mm);
            if (tn * tm > most || (tn * tm == most && waste < most_waste)) {
                most = tn * tm;
                most_waste = waste;
                best = i;
            }
        }
        // ... and split-K raised until the compute units are covered, keeping
        // at least two 128-wide k-steps per split.
        for (int s : kSplitSet) {
            if (s == 1) continue;
            if (k_steps / s < 2) break;
            split = s;
            if (most * s >= cus) break;
        }
    }
    plan->kind = kind;
    plan->tile = best;
    plan->split_k = split;
    return complete_plan(kind, m, n, k_steps, plan);
}

}  // namespace nmspmm
