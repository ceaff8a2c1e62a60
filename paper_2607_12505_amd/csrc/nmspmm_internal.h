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
constexpr int kVBlock = 1024;    // bytes of the 4:2 operand values per (fragment, k-step)
constexpr int kMBlock = 256;     // bytes of the 4:2 operand positions per (fragment, k-step)
constexpr int kThreads = 256;    // threads of a k-sliced workgroup (4 waves of 64)

// Per-lane bytes of a packed block (include/nmspmm.h): value bytes VB and
// position bytes MB of one lane of one (16-row fragment, k-step) block, for
// every layout but DENSE; and the values per window of a mask layout.
constexpr int layout_mask_values(int lay) {
    return lay == NM_LAYOUT_MK3 ? 3 : lay == NM_LAYOUT_MK4 ? 4 : lay == NM_LAYOUT_MK5 ? 5 : 0;
}
constexpr int layout_lane_vbytes(int lay) {
    return lay == NM_LAYOUT_SP42 ? 16 : lay == NM_LAYOUT_C14 ? 8 : lay == NM_LAYOUT_C18 ? 4 : lay == NM_LAYOUT_C28 ? 8
                                                                                             : 4 * layout_mask_values(lay);
}
constexpr int layout_lane_mbytes(int lay) {
    return lay == NM_LAYOUT_C14 || lay == NM_LAYOUT_C18 ? 2 : 4;
}
// Kernel families whose weight operand is the structured-sparse 4:2 form
// (the others run the dense matrix instruction on a dense weight tile).
constexpr bool kind_is_sp42(int kind) {
    return kind == NM_KIND_SP42 || kind == NM_KIND_C14 || kind == NM_KIND_C18 || kind == NM_KIND_C28;
}
constexpr bool kind_is_valid(int kind) { return kind >= NM_KIND_SP42 && kind <= NM_KIND_MK5; }

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
    {2, 2, 4, 5, 2, kOutSplit},  // 11: 128 ch x 160 tok, 2-slot ring (long reductions, narrow outputs)
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
    // Workgroups gemm_grid .. gridDim.x - 1 of the launch do not belong to the
    // GEMM: they expand another compact weight (x_kind, blocks as in the
    // packed layout) into x_out, one block per wave (nm_spmm_out_expand).
    int gemm_grid = 0x7fffffff;
    int x_kind = 0;
    const int8_t *x_vals = nullptr;
    const uint8_t *x_meta = nullptr;
    int8_t *x_out = nullptr;
    int x_n = 0, x_k = 0, x_blocks = 0, x_k_steps = 0;
};

// Workspace of a plan: with split_k > 1 a fixed block of per-tile arrival
// counters, then split_k partial [m x n] int32 tiles; then, with expand = 1,
// the expanded weight.  The counter block never overlaps partial sums or an
// expanded weight, whatever the plan, so counters left at zero by one call
// are still zero for the next call with another plan.
constexpr size_t kCounterBytes = 16384;
constexpr int kMaxSplitTiles = (int)(kCounterBytes / 4);
// Static scratch of nm_spmm_noalloc: the counter block plus 32 MiB of partial
// tiles, held by every device the library runs on until the process ends.
constexpr size_t kNoAllocScratchBytes = kCounterBytes + ((size_t)32 << 20);
size_t split_workspace_bytes(int split_k, int m, int n);     // counters + partials (0 without split)
size_t expand_offset(int split_k, int m, int n);             // where the expanded weight starts
size_t workspace_bytes(const nm_plan &plan, int m, int n);   // the whole workspace of a completed plan

// Expansion of a compact weight once per call (plan.expand == 1): the kernel
// family that then runs, and the bytes of the expanded weight (the 4:2
// operand, 1280 bytes per fragment and k-step, or dense W [n x k]).
constexpr bool kind_is_compact(int kind) { return kind != NM_KIND_SP42 && kind != NM_KIND_DENSE && kind_is_valid(kind); }
constexpr int expanded_kind(int kind) { return kind_is_sp42(kind) ? NM_KIND_SP42 : NM_KIND_DENSE; }
int64_t expanded_bytes(int kind, int n, int k);
int launch_expand(int kind, const int8_t *vals, const uint8_t *meta, int n, int k, int8_t *out, void *stream);
// Waves per workgroup of a tile's kernel (each tail workgroup of a launch
// that carries an expansion expands one block per wave).
constexpr int tile_waves(const TileCfg &t) { return t.layout == kKSliced ? kThreads / 64 : t.wn * t.wm; }

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
                   const nm_plan *forced, WorkspaceFn ws_fn, const nm_expand_job *job = nullptr);
nm_status check_desc(const nm_desc *d);
int kind_of(const nm_desc *d);

// Planner shared by both GEMM families.
nm_status make_plan(int kind, int m, int n, int k, int out_mode, nm_plan *plan);
nm_status complete_plan(int kind, int m, int n, int k, nm_plan *plan);

}  // namespace nmspmm
