// Internal declarations shared by the host files and the kernels of libnmspmm.
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime.h>

#include "../../include/nmspmm.h"

namespace nmspmm {

// Fixed geometry of the packed weight and of the matrix instructions.
constexpr int kFragRows = 16;    // rows (output channels) per MFMA fragment
constexpr int kKStep = 128;      // dense-equivalent k per structured-sparse MFMA
constexpr int kVBlock = 1024;    // packed value bytes per (fragment, k-step, stream)
constexpr int kMBlock = 256;     // packed position bytes per (fragment, k-step, stream)
constexpr int kThreads = 256;    // threads of a k-sliced workgroup (4 waves of 64)

// Kernel layouts of a workgroup tile.
//   kOutSplit:  WN x WM waves (4 or 8), each owning FN x FM fragments of
//               16 x 16 outputs (tile_n = WN * FN * 16 channels, tile_m = WM *
//               FM * 16 tokens); one output tile per workgroup.
//   kKSliced:   every wave computes the whole FN x FM-fragment tile over a
//               quarter of the k-steps (wn = wm = 1); one tile per workgroup.
// nst = depth of the ring of k-step slots staged in LDS.
enum Layout { kOutSplit = 0, kKSliced = 1 };

struct TileCfg {
    int wn, wm, fn, fm, nst, layout;
    constexpr int tile_n() const { return wn * fn * kFragRows; }
    constexpr int tile_m() const { return wm * fm * 16; }
};

// Tiles the kernels are instantiated for: the candidates of the planner
// (each is its choice for some class of shapes).
constexpr TileCfg kTiles[] = {
    {2, 2, 4, 4, 2, kOutSplit},  // 0: 128 ch x 128 tok, 2-slot ring (3 workgroups per CU)
    {2, 2, 4, 2, 2, kOutSplit},  // 1: 128 ch x  64 tok, 2-slot ring
    {2, 2, 2, 4, 2, kOutSplit},  // 2:  64 ch x 128 tok, 2-slot ring
    {2, 2, 2, 2, 2, kOutSplit},  // 3:  64 ch x  64 tok, 2-slot ring
    {2, 4, 8, 4, 3, kOutSplit},  // 4: 256 ch x 256 tok, 8 waves (2 x 4), 3-slot ring
    {2, 2, 4, 1, 2, kOutSplit},  // 5: 128 ch x  32 tok, 2-slot ring
    {4, 2, 2, 4, 2, kOutSplit},  // 6: 128 ch x 128 tok, 8 waves (4 x 2), 2-slot ring
    {1, 1, 4, 4, 3, kKSliced},   // 7:  64 ch x  64 tok, k-sliced over the waves
    {1, 1, 2, 4, 3, kKSliced},   // 8:  32 ch x  64 tok, k-sliced
    {1, 1, 4, 2, 3, kKSliced},   // 9:  64 ch x  32 tok, k-sliced
    {1, 1, 2, 2, 3, kKSliced},   // 10: 32 ch x  32 tok, k-sliced
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);
constexpr size_t kLdsPerCu = 160 * 1024;

// Everything a GEMM kernel needs; passed by value as the kernel argument.
struct GemmArgs {
    const int8_t *X;        // [m x k] row-major
    const int8_t *A;        // packed values (sparse kinds) or W [n x k] (dense)
    const uint8_t *meta;    // packed positions (sparse kinds)
    int32_t *Y;             // [m x n] or null
    uint16_t *Yh;           // [m x n] or null
    const float *scale;     // [n] (needed with Yh)
    int8_t *Yq;             // [m x n] or null
    const float *qscale;    // [n] (needed with Yq)
    int32_t *counters;      // one per output tile (split_k > 1)
    int32_t *partials;      // [split_k x m x n] (split_k > 1)
    int m, n, k;
    int k_steps, n_frags;
    int tiles_n, tiles_m, split_k;
    int group_rows;         // tile order: 0 row by row, else groups of this many tile rows
};

// Workspace of a split-K plan: a fixed block of per-tile arrival counters,
// then split_k partial [m x n] int32 tiles.  The counter block never overlaps
// partial sums, whatever the plan, so counters left at zero by one call are
// still zero for the next call with another plan.
constexpr size_t kCounterBytes = 16384;
constexpr int kMaxSplitTiles = (int)(kCounterBytes / 4);
// Static scratch of nm_spmm_noalloc: the counter block plus 32 MiB of partial
// tiles, held by every device the library runs on until the process ends.
constexpr size_t kNoAllocScratchBytes = kCounterBytes + ((size_t)32 << 20);
size_t workspace_bytes(int split_k, int tiles, int m, int n);

int device_cu_count();     // cached per device; 256 when no device is visible

// Launches the kernel of (kind, tile) on the stream.  Returns a hipError_t value.
int launch_gemm(int kind, int tile, const GemmArgs &args, int grid, void *stream);
int launch_zero(void *ptr, size_t bytes, void *stream);
int launch_quantize_f16(const uint16_t *x, int64_t count, float inv_scale, int8_t *xq, void *stream);

// Argument checks, planning and launch of one GEMM (nmspmm_api.cpp).  When
// the plan needs a workspace and ws_fn is given, ws_fn supplies it instead of
// ws / ws_bytes.
typedef nm_status (*WorkspaceFn)(size_t need, void *stream, void **ws, size_t *ws_bytes);
nm_status run_gemm(int kind, const int8_t *X, int m, const int8_t *A, const uint8_t *meta, int n, int k,
                   int k_steps, int n_frags, const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                   const nm_plan *forced, WorkspaceFn ws_fn);
nm_status check_desc(const nm_desc *d);
int kind_of(const nm_desc *d);

// Planner shared by both GEMM families.
nm_status make_plan(int kind, int m, int n, int k_steps, int out_mode, nm_plan *plan);
nm_status complete_plan(int kind, int m, int n, int k_steps, nm_plan *plan);

}  // namespace nmspmm
