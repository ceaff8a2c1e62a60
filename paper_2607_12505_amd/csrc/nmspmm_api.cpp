// C ABI entry points: argument checks, planning and dispatch (host only).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

#include "nmspmm_internal.h"

using namespace nmspmm;

namespace {

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int out_mode_of(const nm_outputs &o) {
    return (o.y ? NM_OUT_I32 : 0) | (o.yh ? NM_OUT_F16 : 0) | (o.yq ? NM_OUT_I8 : 0);
}

nm_outputs outputs_of(int32_t *Y, const float *scale, uint16_t *Yh) {
    nm_outputs o;
    o.y = Y;
    o.yh = Yh;
    o.scale = scale;
    o.yq = nullptr;
    o.qscale = nullptr;
    return o;
}

// Tile order of the launch.  Row by row, the tiles in flight on one XCD share
// two or three rows of X and sweep the whole weight; when X arrives cold from
// HBM -- as it does inside a network's sequence of layers, where the layers
// before have streamed far more than the last-level cache holds -- all of
// them wait on the same few rows, one k-step at a time.  Walking groups of 16
// tile rows column by column puts 16 distinct rows of X in flight per XCD
// (2 MB of X and a few column tiles of the weight stay in its 4 MB L2).  Timed
// with a 75 MB read before every launch (ViT-L/16-384 batch 32, m = 18464):
// 2:4 fc1 on 128 x 128 tiles 125 -> 82-86 us, qkv 93 -> 65-68, fc2 84 -> 77-79,
// proj 36 -> 32; groups of 4 or 8 rows gained less, 32 lost.  Launches with
// fewer than 32 rows of tiles keep the row order.
constexpr int kGroupRows = 16;

int64_t stored_weight_bytes(int kind, int n, int k, int n_frags, int k_steps) {
    return kind == NM_KIND_DENSE ? (int64_t)n * k
                                 : (int64_t)n_frags * k_steps * 64 * (layout_lane_vbytes(kind) + layout_lane_mbytes(kind));
}

int group_rows_for(int tiles_m) { return tiles_m >= 2 * kGroupRows ? kGroupRows : 0; }

// Whether the byte ranges [a, a + na) and [b, b + nb) intersect (a null or
// empty range intersects nothing).
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
    if (!a || !b || na <= 0 || nb <= 0) return false;
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

}  // namespace

namespace nmspmm {

// Checks an expansion job before anything is launched.
static nm_status check_job(const nm_expand_job *job) {
    nm_desc e;
    size_t need = 0;
    nm_status st = nm_expand_size(job->desc, &e, &need);
    if (st != NM_OK) return st;
    if (!job->vals || !job->meta || !job->out || !aligned16(job->vals) || !aligned16(job->meta) ||
        !aligned16(job->out))
        return NM_ERR_ARG;
    return job->out_bytes < need ? NM_ERR_WORKSPACE : NM_OK;
}

nm_status run_gemm(int kind, const int8_t *X, int m, const int8_t *A, const uint8_t *meta, int n, int k,
                   int k_steps, int n_frags, const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                   const nm_plan *forced, WorkspaceFn ws_fn, const nm_expand_job *job) {
    if (m < 0) return NM_ERR_SHAPE;
    if (job) {
        nm_status st = check_job(job);
        if (st != NM_OK) return st;
    }
    if (m == 0) {
        // nothing to compute (empty tensors may carry null pointers); a job still runs
        if (!job) return NM_OK;
        const nm_desc *d = job->desc;
        return launch_expand(kind_of(d), job->vals, job->meta, d->n, d->k, job->out, stream) == 0 ? NM_OK : NM_ERR_HIP;
    }
    if (!out) return NM_ERR_ARG;
    const nm_outputs o = *out;
    if (!X || !A || (kind != NM_KIND_DENSE && !meta)) return NM_ERR_ARG;
    if (!o.y && !o.yh && !o.yq) return NM_ERR_ARG;
    if ((o.yh && !o.scale) || (o.yq && !o.qscale)) return NM_ERR_ARG;
    if (!aligned16(X) || !aligned16(A) || (meta && !aligned16(meta)) || (o.y && !aligned16(o.y)) ||
        (o.yh && !aligned16(o.yh)) || (o.yh && !aligned16(o.scale)) || (o.yq && !aligned16(o.yq)) ||
        (o.yq && !aligned16(o.qscale)))
        return NM_ERR_ARG;
    // outputs, X and the weight are addressed with 32-bit byte offsets
    if ((int64_t)m * n >= ((int64_t)1 << 29)) return NM_ERR_SHAPE;
    if ((int64_t)m * k >= ((int64_t)1 << 32)) return NM_ERR_SHAPE;
    if (stored_weight_bytes(kind, n, k, n_frags, k_steps) >= ((int64_t)1 << 32)) return NM_ERR_SHAPE;
    nm_plan plan;
    if (forced) {
        plan = *forced;
        nm_status st = complete_plan(kind, m, n, k, &plan);
        if (st != NM_OK) return st;
    } else {
        nm_status st = make_plan(kind, m, n, k, out_mode_of(o), &plan);
        if (st != NM_OK) return st;
    }
    const size_t need = workspace_bytes(plan, m, n);
    if (need > 0 && ws_fn) {
        nm_status st = ws_fn(need, stream, &ws, &ws_bytes);
        if (st != NM_OK) return st;
    }
    if (need > 0 && (!ws || ws_bytes < need || !aligned16(ws))) return NM_ERR_WORKSPACE;
    if (job) {
        // the expansion a launch carries writes job->out while the GEMM runs:
        // it may not overlap anything the GEMM reads or writes
        const int64_t jb = (int64_t)job->out_bytes, mn = (int64_t)m * n;
        if (overlaps(job->out, jb, X, (int64_t)m * k) ||
            overlaps(job->out, jb, A, kind == NM_KIND_DENSE ? (int64_t)n * k
                                                            : (int64_t)n_frags * k_steps * 64 * layout_lane_vbytes(kind)) ||
            overlaps(job->out, jb, meta, kind == NM_KIND_DENSE ? 0
                                                               : (int64_t)n_frags * k_steps * 64 * layout_lane_mbytes(kind)) ||
            overlaps(job->out, jb, o.y, 4 * mn) || overlaps(job->out, jb, o.yh, 2 * mn) ||
            overlaps(job->out, jb, o.yq, mn) || overlaps(job->out, jb, ws, (int64_t)need) ||
            overlaps(job->out, jb, job->vals, job->desc->vals_bytes) ||
            overlaps(job->out, jb, job->meta, job->desc->meta_bytes))
            return NM_ERR_ARG;
    }

    // With expand = 1 the compact weight is first expanded into the workspace
    // (after the split-K area), and the 4:2-operand or dense kernel runs on it.
    int run_kind = kind;
    if (plan.expand) {
        int8_t *exp = (int8_t *)ws + expand_offset(plan.split_k, m, n);
        if (launch_expand(kind, A, meta, n, k, exp, stream) != 0) return NM_ERR_HIP;
        run_kind = expanded_kind(kind);
        A = exp;
        meta = run_kind == NM_KIND_SP42 ? (const uint8_t *)(exp + (int64_t)n_frags * k_steps * kVBlock) : nullptr;
    }
    const bool split = plan.split_k > 1;
    GemmArgs a;
    a.X = X;
    a.A = A;
    a.meta = meta;
    a.Y = o.y;
    a.Yh = o.yh;
    a.scale = o.scale;
    a.Yq = o.yq;
    a.qscale = o.qscale;
    a.counters = split ? (int32_t *)ws : nullptr;
    a.partials = split ? (int32_t *)((char *)ws + kCounterBytes) : nullptr;
    a.m = m;
    a.n = n;
    a.k = k;
    a.k_steps = k_steps;
    a.n_frags = n_frags;
    a.tiles_n = (n + plan.tile_n - 1) / plan.tile_n;
    a.tiles_m = (m + plan.tile_m - 1) / plan.tile_m;
    a.split_k = plan.split_k;
    a.group_rows = group_rows_for(a.tiles_m);
    a.gemm_grid = plan.grid;
    int grid = plan.grid;
    if (job) {
        // the job's blocks go to workgroups appended after the GEMM's, one per wave
        const nm_desc *d = job->desc;
        const int per = tile_waves(kTiles[plan.tile]);
        const int64_t blocks = (int64_t)d->n_frags * d->k_steps;
        const int64_t extra = (blocks + per - 1) / per;
        if ((int64_t)grid + extra > 0x7fffffff) return NM_ERR_SHAPE;
        a.x_kind = kind_of(d);
        a.x_vals = job->vals;
        a.x_meta = job->meta;
        a.x_out = job->out;
        a.x_n = d->n;
        a.x_k = d->k;
        a.x_blocks = (int)blocks;
        a.x_k_steps = d->k_steps;
        grid += (int)extra;
    }
    int err = launch_gemm(run_kind, plan.tile, a, grid, stream);
    return err == 0 ? NM_OK : NM_ERR_HIP;
}

nm_status check_desc(const nm_desc *d) {
    if (!d) return NM_ERR_ARG;
    nm_desc chk;
    if (nm_compress_size(d->n, d->k, d->nm_n, d->nm_m, &chk) != NM_OK) return NM_ERR_ARG;
    if (chk.kind != d->kind || chk.layout != d->layout || chk.n_frags != d->n_frags || chk.k_steps != d->k_steps ||
        chk.vals_bytes != d->vals_bytes || chk.meta_bytes != d->meta_bytes)
        return NM_ERR_ARG;
    return NM_OK;
}

int kind_of(const nm_desc *d) { return d->kind; }

}  // namespace nmspmm

extern "C" const char *nm_status_string(nm_status s) {
    switch (s) {
        case NM_OK: return "ok";
        case NM_ERR_ARG: return "invalid argument";
        case NM_ERR_SHAPE: return "unsupported shape";
        case NM_ERR_PATTERN: return "weight violates the N:M pattern";
        case NM_ERR_UNSUPPORTED: return "unsupported N:M pattern";
        case NM_ERR_WORKSPACE: return "workspace missing or too small";
        case NM_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

extern "C" int nm_num_tiles(void) { return kNumTiles; }

extern "C" nm_status nm_tile_info(int tile, int *tile_n, int *tile_m) {
    if (tile < 0 || tile >= kNumTiles || !tile_n || !tile_m) return NM_ERR_ARG;
    *tile_n = kTiles[tile].tile_n();
    *tile_m = kTiles[tile].tile_m();
    return NM_OK;
}

extern "C" nm_status nm_plan_kernel_name(const nm_plan *plan, char *buf, int len) {
    if (!plan || !buf || len <= 0 || plan->tile < 0 || plan->tile >= kNumTiles) return NM_ERR_ARG;
    if (!kind_is_valid(plan->kind)) return NM_ERR_ARG;
    const TileCfg &t = kTiles[plan->tile];
    const int kind = plan->expand == 1 && kind_is_compact(plan->kind) ? expanded_kind(plan->kind) : plan->kind;
    int w;
    if (t.layout == kKSliced)
        w = std::snprintf(buf, (size_t)len, "k_gemm_ks<%d, %d, %d, %d>", kind, t.fn, t.fm, t.nst);
    else
        w = std::snprintf(buf, (size_t)len, "k_gemm<%d, %d, %d, %d, %d, %d>", kind, t.wn, t.wm, t.fn, t.fm, t.nst);
    return (w > 0 && w < len) ? NM_OK : NM_ERR_ARG;
}

extern "C" nm_status nm_spmm_plan(const nm_desc *desc, int m, int out_mode, nm_plan *plan) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    return make_plan(kind_of(desc), m, desc->n, desc->k, out_mode, plan);
}

extern "C" nm_status nm_spmm_plan_complete(const nm_desc *desc, int m, nm_plan *plan) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    if (!plan || m < 0) return NM_ERR_ARG;
    return complete_plan(kind_of(desc), m, desc->n, desc->k, plan);
}

extern "C" nm_status nm_gemm_i8_dense_plan(int m, int n, int k, int out_mode, nm_plan *plan) {
    if (n < 1 || k < 1) return NM_ERR_ARG;
    if (k % 16 != 0 || n % 4 != 0) return NM_ERR_SHAPE;
    return make_plan(NM_KIND_DENSE, m, n, k, out_mode, plan);
}

extern "C" nm_status nm_workspace_size(const nm_plan *plan, int m, int n, size_t *bytes) {
    if (!plan || !bytes || m < 0 || n < 1 || plan->split_k < 1 || plan->tile < 0 || plan->tile >= kNumTiles ||
        (plan->expand != 0 && plan->expand != 1) || plan->expand_bytes < 0)
        return NM_ERR_ARG;
    *bytes = workspace_bytes(*plan, m, n);
    return NM_OK;
}

extern "C" nm_status nm_workspace_init(void *ws, size_t bytes, void *stream) {
    if (bytes == 0) return NM_OK;
    if (!ws || !aligned16(ws)) return NM_ERR_ARG;
    return launch_zero(ws, bytes, stream) == 0 ? NM_OK : NM_ERR_HIP;
}

extern "C" nm_status nm_spmm_out(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                                 const nm_desc *desc, const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                                 const nm_plan *plan) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    return run_gemm(kind_of(desc), X, m, vals, meta, desc->n, desc->k, desc->k_steps, desc->n_frags, out, ws,
                    ws_bytes, stream, plan, nullptr);
}

extern "C" nm_status nm_spmm_out_expand(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                                        const nm_desc *desc, const nm_outputs *out, void *ws, size_t ws_bytes,
                                        void *stream, const nm_plan *plan, const nm_expand_job *job) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    return run_gemm(kind_of(desc), X, m, vals, meta, desc->n, desc->k, desc->k_steps, desc->n_frags, out, ws,
                    ws_bytes, stream, plan, nullptr, job);
}

extern "C" nm_status nm_spmm_ex(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                                const nm_desc *desc, int32_t *Y, const float *scale, uint16_t *Yh,
                                void *ws, size_t ws_bytes, void *stream, const nm_plan *plan) {
    const nm_outputs o = outputs_of(Y, scale, Yh);
    return nm_spmm_out(X, m, vals, meta, desc, &o, ws, ws_bytes, stream, plan);
}

extern "C" nm_status nm_spmm(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                             const nm_desc *desc, int32_t *Y, const float *scale, uint16_t *Yh,
                             void *ws, size_t ws_bytes, void *stream) {
    return nm_spmm_ex(X, m, vals, meta, desc, Y, scale, Yh, ws, ws_bytes, stream, nullptr);
}

extern "C" nm_status nm_gemm_i8_dense_out(const int8_t *X, int m, const int8_t *W, int n, int k,
                                          const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                                          const nm_plan *plan) {
    if (n < 1 || k < 1) return NM_ERR_ARG;
    if (k % 16 != 0 || n % 4 != 0) return NM_ERR_SHAPE;
    const int k_steps = (k + kKStep - 1) / kKStep;
    return run_gemm(NM_KIND_DENSE, X, m, W, nullptr, n, k, k_steps, (n + kFragRows - 1) / kFragRows, out, ws,
                    ws_bytes, stream, plan, nullptr);
}

extern "C" nm_status nm_gemm_i8_dense_out_expand(const int8_t *X, int m, const int8_t *W, int n, int k,
                                                 const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                                                 const nm_plan *plan, const nm_expand_job *job) {
    if (n < 1 || k < 1) return NM_ERR_ARG;
    if (k % 16 != 0 || n % 4 != 0) return NM_ERR_SHAPE;
    const int k_steps = (k + kKStep - 1) / kKStep;
    return run_gemm(NM_KIND_DENSE, X, m, W, nullptr, n, k, k_steps, (n + kFragRows - 1) / kFragRows, out, ws,
                    ws_bytes, stream, plan, nullptr, job);
}

extern "C" nm_status nm_gemm_i8_dense_ex(const int8_t *X, int m, const int8_t *W, int n, int k,
                                         int32_t *Y, const float *scale, uint16_t *Yh,
                                         void *ws, size_t ws_bytes, void *stream, const nm_plan *plan) {
    const nm_outputs o = outputs_of(Y, scale, Yh);
    return nm_gemm_i8_dense_out(X, m, W, n, k, &o, ws, ws_bytes, stream, plan);
}

extern "C" nm_status nm_gemm_i8_dense(const int8_t *X, int m, const int8_t *W, int n, int k,
                                      int32_t *Y, const float *scale, uint16_t *Yh,
                                      void *ws, size_t ws_bytes, void *stream) {
    return nm_gemm_i8_dense_ex(X, m, W, n, k, Y, scale, Yh, ws, ws_bytes, stream, nullptr);
}

extern "C" nm_status nm_expand_size(const nm_desc *desc, nm_desc *expanded, size_t *bytes) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    if (!expanded || !bytes) return NM_ERR_ARG;
    const int kind = kind_of(desc);
    if (!kind_is_compact(kind)) return NM_ERR_ARG;
    // the expanded form is the packed form of 2:4 (4:2-operand kinds) or of a
    // dense pattern (mask kinds) for the same shape
    const bool sp = expanded_kind(kind) == NM_KIND_SP42;
    st = nm_compress_size(desc->n, desc->k, sp ? 2 : 8, sp ? 4 : 8, expanded);
    if (st != NM_OK) return st;
    if (expanded->vals_bytes + expanded->meta_bytes != expanded_bytes(kind, desc->n, desc->k)) return NM_ERR_ARG;
    *bytes = (size_t)(expanded->vals_bytes + expanded->meta_bytes);
    return NM_OK;
}

extern "C" nm_status nm_expand(const nm_desc *desc, const int8_t *vals, const uint8_t *meta, int8_t *out,
                               size_t out_bytes, void *stream) {
    nm_desc e;
    size_t need = 0;
    nm_status st = nm_expand_size(desc, &e, &need);
    if (st != NM_OK) return st;
    if (!vals || !meta || !out || !aligned16(vals) || !aligned16(meta) || !aligned16(out)) return NM_ERR_ARG;
    if (out_bytes < need) return NM_ERR_WORKSPACE;
    return launch_expand(kind_of(desc), vals, meta, desc->n, desc->k, out, stream) == 0 ? NM_OK : NM_ERR_HIP;
}

extern "C" nm_status nm_quantize_f16(const uint16_t *x, int64_t count, float inv_scale, int8_t *xq, void *stream) {
    if (count < 0) return NM_ERR_SHAPE;
    if (count == 0) return NM_OK;
    if (!x || !xq || !aligned16(x) || !aligned16(xq)) return NM_ERR_ARG;
    return launch_quantize_f16(x, count, inv_scale, xq, stream) == 0 ? NM_OK : NM_ERR_HIP;
}
