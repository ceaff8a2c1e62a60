// Internal declarations shared by the host files and the kernels of libnmspmm.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/nmspmm.h"

namespace nmspmm {

// Fixed geometry of the packed weight and of the matrix instructions.
constexpr int kFragRows = 16;    // rows (output channels) per MFMA fragment
constexpr int kKStep = 128;      // dense-equivalent k per structured-sparse MFMA
constexpr int kVBlock = 1024;    // packed value bytes per (fragment, k-step, stream)
constexpr int kMBlock = 256;     // packed position bytes per (fragment, k-step, stream)
constexpr int kThreads = 256;    // threads per workgroup (4 waves of 64)

// Workgroup tile: WN x WM waves, each owning FN x FM fragments of 16 x 16
// outputs.  tile_n = WN * FN * 16 channels, tile_m = WM * FM * 16 tokens.
struct TileCfg {
    int wn, wm, fn, fm;
    constexpr int tile_n() const { return wn * fn * kFragRows; }
    constexpr int tile_m() const { return wm * fm * 16; }
};

// Tiles the kernels are instantiated for, from the largest to the smallest.
constexpr TileCfg kTiles[] = {
    {2, 2, 4, 4},  // 0: 128 ch x 128 tok
    {4, 1, 4, 4},  // 1: 256 ch x  64 tok
    {1, 4, 4, 4},  // 2:  64 ch x 256 tok
    {2, 2, 4, 2},  // 3: 128 ch x  64 tok
    {2, 2, 2, 4},  // 4:  64 ch x 128 tok
    {2, 2, 2, 2},  // 5:  64 ch x  64 tok
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

// Everything a GEMM kernel needs; passed by value as the kernel argument.
struct GemmArgs {
    const int8_t *X;        // [m x k] row-major
    const int8_t *A;        // packed values (sparse kinds) or W [n x k] (dense)
    const uint8_t *meta;    // packed positions (sparse kinds)
    int32_t *Y;             // [m x n] or null
    uint16_t *Yh;           // [m x n] or null
    const float *scale;     // [n] (needed with Yh)
    int32_t *counters;      // one per output tile (split_k > 1)
    int32_t *partials;      // [split_k x m x n] (split_k > 1)
    int m, n, k;
    int k_steps, n_frags;
    int tiles_n, tiles_m, split_k;
};

// Workspace of a split-K plan: a fixed block of per-tile arrival counters,
// then split_k partial [m x n] int32 tiles.  The counter block never overlaps
// partial sums, whatever the plan, so counters left at zero by one call are
// still zero for the next call with another plan.
constexpr size_t kCounterBytes = 16384;
constexpr int kMaxSplitTiles = (int)(kCounterBytes / 4);
size_t workspace_bytes(int split_k, int tiles, int m, int n);

int device_cu_count();     // cached per device; 256 when no device is visible

// Launches the kernel of (kind, tile) on the stream.  Returns a hipError_t value.
int launch_gemm(int kind, int tile, const GemmArgs &args, int grid, void *stream);
int launch_zero(void *ptr, size_t bytes, void *stream);

// Planner shared by both GEMM families.
nm_status make_plan(int kind, int m, int n, int k_steps, int out_mode, nm_plan *plan);
nm_status complete_plan(int kind, int m, int n, int k_steps, nm_plan *plan);

}  // namespace nmspmm
