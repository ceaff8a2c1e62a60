/*
 * nmspmm.h -- C ABI of libnmspmm: N:M sparse INT8 GEMM for AMD Instinct
 * MI355X (gfx950).
 *
 * The operation (paper: "Realizable N:M Sparse Transformer Inference via
 * Search-Kernel Co-Design"; N:M sparsity Sec. 2.1, MD-SpMM Sec. 4):
 *
 *     Y[i][j] = sum_t X[i][t] * W[j][t]          (exact, int32)
 *     Yh[i][j] = fp16( fp32(Y[i][j]) * scale[j] ) (optional dequantisation)
 *     Yq[i][j] = q8( fp32(Y[i][j]) * qscale[j] )  (optional requantisation)
 *
 * X is int8 [m x k] row-major (m tokens, k = in_features), W is int8 [n x k]
 * row-major (n = out_features, the layout of a PyTorch Linear weight) with at
 * most N nonzeros in every aligned window of M consecutive entries along k.
 * Y is int32 [m x n] row-major, Yh binary16 [m x n] row-major.
 *
 * Conventions for every entry point:
 *   - Every buffer is owned by the caller.  The library never allocates device
 *     memory and never frees anything it is given.  (The one device array the
 *     library owns is the fixed scratch of nm_spmm_noalloc, part of its code
 *     object's static data.)
 *   - "host" pointers are ordinary CPU memory; "device" pointers are GPU
 *     memory of the current HIP device (hipMalloc or a PyTorch CUDA tensor).
 *   - Device pointers must be 16-byte aligned.
 *   - GEMM entry points are asynchronous: they enqueue kernels on `stream`
 *     (a hipStream_t; NULL means the default stream) and return.  A status of
 *     NM_OK means the arguments were valid and the launch was accepted; faults
 *     inside a kernel surface at the next synchronising HIP call.
 *   - On any error status nothing has been written to any caller buffer
 *     (except the diagnostic fields of an nm_desc).
 *   - The library has no global mutable state besides a thread-safe cache of
 *     per-device properties and, per device, the scratch array of
 *     nm_spmm_noalloc with its looked-up address.
 */
#ifndef NMSPMM_H
#define NMSPMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum nm_status {
    NM_OK = 0,
    NM_ERR_ARG = 1,          /* null pointer, misaligned pointer, bad plan, negative size */
    NM_ERR_SHAPE = 2,        /* k % M != 0, k % 16 != 0, n % 4 != 0, size too large */
    NM_ERR_PATTERN = 3,      /* a window of W holds more than N nonzeros */
    NM_ERR_UNSUPPORTED = 4,  /* (N, M) outside {1..4}:4 and {1..8}:8 */
    NM_ERR_WORKSPACE = 5,    /* workspace missing or smaller than required */
    NM_ERR_HIP = 6           /* a HIP call (launch, device query) failed */
} nm_status;

/* Output selection bits (used by the planners and workspace queries). */
#define NM_OUT_I32 1
#define NM_OUT_F16 2
#define NM_OUT_I8 4
/* Planner hint (may be or-ed into the out_mode of nm_spmm_plan): the caller
 * runs any once-per-call expansion the plan asks for in an earlier launch
 * (nm_spmm_out_expand), so the expansion costs no launch of its own. */
#define NM_PLAN_EXPAND_CARRIED 8

/* Physical layouts of the packed weight produced by nm_compress, and the
 * kernel families they feed (nm_desc.layout, nm_desc.kind, nm_plan.kind; a
 * layout and its kernel family share a number). */
#define NM_LAYOUT_SP42 1   /* 2:4: the 4:2 operand of the structured-sparse MFMA as stored */
#define NM_LAYOUT_C14 2    /* 1:4: one value and a 2-bit position per 4-group */
#define NM_LAYOUT_DENSE 3  /* W itself, row-major (3:4, 4:4, 6:8, 7:8, 8:8) */
#define NM_LAYOUT_C18 4    /* 1:8: one value and a 3-bit position per 8-window */
#define NM_LAYOUT_C28 5    /* 2:8: two values and two 3-bit positions per 8-window */
#define NM_LAYOUT_MK3 6    /* 3:8: three values and an 8-bit occupancy mask per 8-window */
#define NM_LAYOUT_MK4 7    /* 4:8: four values and an 8-bit occupancy mask per 8-window */
#define NM_LAYOUT_MK5 8    /* 5:8: five values and an 8-bit occupancy mask per 8-window */

/*
 * Descriptor of a packed weight.  Filled by nm_compress / nm_compress_size and
 * treated as read-only afterwards.
 *
 * The paper's packed form B_pack keeps each window's nonzero values together
 * with their positions inside the window (Sec. 4.2).  In memory it is compact:
 * N/M of the values plus a few position bits per window; the GEMM kernels
 * expand it on the fly -- into the 4:2 operand of the gfx950 structured-sparse
 * matrix instruction (two (value, 2-bit position) slots per aligned 4-group of
 * k) for the patterns with at most 2 nonzeros in every 4-group, or into a dense
 * tile for the dense matrix instruction for 3:8, 4:8 and 5:8.  Patterns whose
 * compact form would save too little (3:4, 4:4, 6:8, 7:8, 8:8) keep W as it is.
 *
 * Canonical slots (SP42, C14, C18, C28): a window (or 4-group) of M weights
 * with S slots holds its nonzeros by ascending position, then zero-valued
 * padding at the smallest unused positions; the S positions are sorted
 * ascending.  Mask layouts (MKn) hold a window's nonzeros by ascending
 * position, then zeros, and bit p of the window's mask is set iff position p
 * is nonzero.
 *
 * Every layout except DENSE is a sequence of blocks, one per (16-row fragment
 * f, 128-wide k-step s), block b = f * S + s with F = ceil(n / 16) fragments
 * and S = ceil(k / 128) k-steps.  Lane L (0..63) of block b covers row
 * r = 16 f + L % 16 and the 32 columns starting at c0 = 128 s + 32 (L / 16);
 * "group g" is W[r][c0 + 4g .. +4) (g = 0..7) and "window w" is
 * W[r][c0 + 8w .. +8) (w = 0..3).  With VB value bytes and MB position bytes
 * per lane, lane L's bytes are vals[(64 b + L) * VB ..] and
 * meta[(64 b + L) * MB ..] (little endian):
 *
 *   SP42 (VB 16, MB 4):  vals[.. + 2g + t] = slot t of group g (2 slots);
 *                        meta bits [4g + 2t + 1 : 4g + 2t] = its position 0..3
 *   C14  (VB 8, MB 2):   vals[.. + g] = slot of group g (1 slot);
 *                        meta bits [2g + 1 : 2g] = its position 0..3
 *   C18  (VB 4, MB 2):   vals[.. + w] = slot of window w (1 slot);
 *                        meta bits [3w + 2 : 3w] = its position 0..7, bits 12..15 zero
 *   C28  (VB 8, MB 4):   vals[.. + 2w + t] = slot t of window w (2 slots);
 *                        meta bits [6w + 3t + 2 : 6w + 3t] = its position 0..7, bits 24..31 zero
 *   MKn  (VB 4n, MB 4):  vals[.. + n w + j] = the j-th nonzero of window w (0 past the last);
 *                        meta byte w = the occupancy mask of window w
 *
 * Rows >= n and columns >= k are zero.  vals_bytes = 64 F S VB and
 * meta_bytes = 64 F S MB: per weight, N/M value bytes and (SP42, C14) exactly
 * the position bits, (C18, C28) the position bits padded to 16 or 32 bits per
 * lane (0.5 and 1 bit per weight against 0.375 and 0.75), (MKn) one mask bit,
 * all rounded up to whole fragments and k-steps.  DENSE: vals = W [n x k]
 * row-major (vals_bytes = n k), meta_bytes = 0 (meta may be NULL).
 */
typedef struct nm_desc {
    int32_t n, k;          /* logical W shape [n x k] */
    int32_t nm_n, nm_m;    /* pattern: at most nm_n nonzeros per aligned window of nm_m */
    int32_t kind;          /* NM_KIND_* of the kernels that consume this layout */
    int32_t layout;        /* NM_LAYOUT_* */
    int32_t n_frags;       /* ceil(n / 16) */
    int32_t k_steps;       /* ceil(k / 128) */
    int64_t vals_bytes;    /* bytes of the packed values */
    int64_t meta_bytes;    /* bytes of the packed positions or masks */
    int32_t bad_row;       /* first offending row when NM_ERR_PATTERN, else -1 */
    int32_t bad_group;     /* its window index (k / nm_m units), else -1 */
} nm_desc;

/*
 * Launch plan of a GEMM (paper Sec. 4.3, adaptive parallelism): a workgroup
 * tile of tile_n output channels x tile_m tokens, and split_k partitions of
 * the reduction axis whose partial sums are merged at the end.  For a compact
 * weight (the C14, C18, C28 and MKn layouts) the plan also says where the
 * weight is expanded: inside every workgroup, one k-step at a time, ahead of
 * its use (expand = 0), or once per call by a separate kernel into the
 * workspace, which the 4:2-operand (C14, C18, C28) or dense (MKn) GEMM kernel
 * then reads (expand = 1): the first costs the expansion once per row of
 * output tiles, the second once per call plus a launch.  Plans come from the
 * planners below; callers may also build one from nm_tile_info to force a
 * schedule.  Every valid plan gives bit-identical results.
 */
typedef struct nm_plan {
    int32_t kind;          /* NM_KIND_* (the weight's kind) */
    int32_t tile;          /* index into the tile table, 0 .. nm_num_tiles()-1 */
    int32_t tile_n;        /* output channels per workgroup (filled by the library) */
    int32_t tile_m;        /* tokens per workgroup (filled by the library) */
    int32_t split_k;       /* 1, 2, 4 or 8 */
    int32_t grid;          /* workgroups of the GEMM kernel (filled by the library) */
    int32_t expand;        /* 0 or 1 (see above); must be 0 for NM_KIND_SP42 and NM_KIND_DENSE */
    int32_t reserved;      /* 0 */
    int64_t expand_bytes;  /* workspace bytes of the expanded weight (filled by the library) */
} nm_plan;

#define NM_KIND_SP42 1     /* structured-sparse MFMA on the stored 4:2 operand (2:4) */
#define NM_KIND_C14 2      /* structured-sparse MFMA, 1:4 expanded in the kernel */
#define NM_KIND_DENSE 3    /* dense MFMA on a plain row-major W */
#define NM_KIND_C18 4      /* structured-sparse MFMA, 1:8 expanded in the kernel */
#define NM_KIND_C28 5      /* structured-sparse MFMA, 2:8 expanded in the kernel */
#define NM_KIND_MK3 6      /* dense MFMA, 3:8 expanded to a dense tile in the kernel */
#define NM_KIND_MK4 7      /* dense MFMA, 4:8 expanded to a dense tile in the kernel */
#define NM_KIND_MK5 8      /* dense MFMA, 5:8 expanded to a dense tile in the kernel */

/* Human-readable name of a status code (static string, never NULL). */
const char *nm_status_string(nm_status s);

/* ---------------------------------------------------------------- packing
 * Offline packing of W into B_pack (Sec. 4.1-4.2; done once before
 * deployment, Sec. 6.1).  Host memory only, synchronous, thread-safe. */

/* Fills desc (shape, layout, sizes) for W [n x k] with pattern nm_n:nm_m
 * without reading any weight.  Errors: NM_ERR_ARG (desc NULL, n or k < 1),
 * NM_ERR_UNSUPPORTED, NM_ERR_SHAPE. */
nm_status nm_compress_size(int n, int k, int nm_n, int nm_m, nm_desc *desc);

/* Packs host W [n x k] (row-major int8) into host buffers vals
 * (desc->vals_bytes) and meta (desc->meta_bytes), and fills desc.
 * Errors: as nm_compress_size, plus NM_ERR_ARG for NULL W/vals/meta and
 * NM_ERR_PATTERN (desc->bad_row / bad_group name the first offending window
 * in row-major order; vals and meta are untouched). */
nm_status nm_compress(const int8_t *W, int n, int k, int nm_n, int nm_m,
                      int8_t *vals, uint8_t *meta, nm_desc *desc);

/* Inverse of nm_compress: writes host W [n x k].  Errors: NM_ERR_ARG for NULL
 * pointers, an inconsistent desc, or packed data that is not in canonical
 * form (two slots of a group at one position holding a nonzero, a nonzero in
 * the padding rows/columns, more nonzeros in a window than nm_n). */
nm_status nm_decompress(const nm_desc *desc, const int8_t *vals, const uint8_t *meta, int8_t *W);

/* ---------------------------------------------------------------- planning */

/* Number of workgroup tiles the kernels are built for, and their sizes. */
int nm_num_tiles(void);
nm_status nm_tile_info(int tile, int *tile_n, int *tile_m);

/* Planner for nm_spmm (Sec. 4.3): picks tile and split_k from
 * (m, n, k, pattern) so that small-token shapes still occupy every compute
 * unit, with split_k from {1, 2, 4, 8}, k-splits on 128-wide k-step
 * boundaries and at least two k-steps per split.  Needs no GPU: without one
 * it assumes 256 compute units.  out_mode is a mask of NM_OUT_* bits, plus
 * NM_PLAN_EXPAND_CARRIED when the caller carries once-per-call expansions in
 * an earlier launch: a compact weight is then expanded once per call (1:4,
 * whose in-kernel decode is cheapest, only with many rows of output-split
 * tiles); without the hint, only GEMMs large enough to amortise a launch of
 * its own expand once per call. */
nm_status nm_spmm_plan(const nm_desc *desc, int m, int out_mode, nm_plan *plan);

/* Completes a plan built by the caller (kind, tile, split_k, expand set) for
 * nm_spmm on this weight and token count: checks it and fills tile_n,
 * tile_m, grid and expand_bytes, so that nm_workspace_size sizes its
 * workspace.  Needs no GPU.  Errors: NM_ERR_ARG (bad descriptor or plan: a
 * kind other than the descriptor's, an unknown tile, split_k outside
 * {1, 2, 4, 8} or above the k-steps, expand = 1 for a kind that is not
 * compact), NM_ERR_SHAPE. */
nm_status nm_spmm_plan_complete(const nm_desc *desc, int m, nm_plan *plan);

/* Same as nm_spmm_plan for the dense baseline GEMM of shape (m, n, k). */
nm_status nm_gemm_i8_dense_plan(int m, int n, int k, int out_mode, nm_plan *plan);

/* Writes into buf (NUL-terminated, at most len bytes) the name of the GEMM
 * kernel template instance a plan launches, e.g. "k_gemm<1, 2, 2, 4, 4, 3>",
 * as it appears in profiler traces (with expand = 1: the 4:2-operand or dense
 * kernel that follows the expansion kernel "k_expand<kind>").  For profiling
 * tools; needs no GPU.
 * Errors: NM_ERR_ARG (bad plan, NULL buf, len too small). */
nm_status nm_plan_kernel_name(const nm_plan *plan, char *buf, int len);

/* Device workspace needed by a plan for an [m x n] output: 0 when split_k == 1
 * and expand == 0; else a 16384-byte block of per-tile counters, followed with
 * split_k > 1 by split_k partial int32 [m x n] tiles, and with expand = 1 by
 * plan->expand_bytes for the expanded weight (256-byte aligned).  A split-K plan may cover at most
 * 4096 output tiles and its partial tiles must total less than 2 GiB.  The
 * planners fill expand_bytes; for a plan built by hand, the GEMM entry points
 * check the workspace against their own sizing.  Errors: NM_ERR_ARG (bad plan
 * or NULL bytes). */
nm_status nm_workspace_size(const nm_plan *plan, int m, int n, size_t *bytes);

/* Zero-fills a workspace on `stream` with a kernel (no memset node, so it
 * may be captured in a HIP graph).  The counter block of a workspace must be
 * zero before its first use; every GEMM call leaves it at zero again, for any
 * plan, so one initialisation per buffer suffices.  Calls that share a
 * workspace must be ordered on one stream (concurrent calls would race on it). */
nm_status nm_workspace_init(void *ws, size_t bytes, void *stream);

/* ---------------------------------------------------------------- GEMMs */

/* Sparse GEMM on a packed weight (Sec. 4.2-4.3): Y = X W^T and/or
 * Yh = fp16(fp32(Y) * scale[j]).
 *   X      device int8 [m x k], row-major (k = desc->k)
 *   vals   device copy of nm_compress's vals (desc->vals_bytes)
 *   meta   device copy of nm_compress's meta (desc->meta_bytes; NULL allowed
 *          when that is 0, i.e. for NM_LAYOUT_DENSE)
 *   desc   host descriptor from nm_compress
 *   Y      device int32 [m x n] or NULL
 *   scale  device float32 [n], required when Yh != NULL, else ignored
 *   Yh     device binary16 bits [m x n] or NULL (Y and Yh may not both be NULL)
 *   ws     device workspace of ws_bytes (nm_workspace_size of the plan;
 *          may be NULL when the plan needs none)
 *   stream hipStream_t or NULL
 * m == 0 is a valid no-op (no pointer is examined, nothing is launched).  Errors: NM_ERR_ARG, NM_ERR_SHAPE (m < 0 or an
 * m·n >= 2^29, m·k >= 2^32 or a weight of 2^32 bytes or more: outputs, X and the
 * weight are addressed with 32-bit byte offsets), NM_ERR_WORKSPACE,
 * NM_ERR_HIP. */
nm_status nm_spmm(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                  const nm_desc *desc, int32_t *Y, const float *scale, uint16_t *Yh,
                  void *ws, size_t ws_bytes, void *stream);

/* nm_spmm with an explicit plan (NULL = the planner's); the plan's kind must
 * be the descriptor's kind (nm_spmm_plan returns such plans). */
nm_status nm_spmm_ex(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                     const nm_desc *desc, int32_t *Y, const float *scale, uint16_t *Yh,
                     void *ws, size_t ws_bytes, void *stream, const nm_plan *plan);

/* Dense INT8 GEMM baseline on the same shapes (the paper compares against a
 * vendor dense GEMM, Sec. 6.1): Y = X W^T with W device int8 [n x k] plain
 * row-major, same outputs, workspace and error rules as nm_spmm; requires
 * k % 16 == 0 and n % 4 == 0. */
nm_status nm_gemm_i8_dense(const int8_t *X, int m, const int8_t *W, int n, int k,
                           int32_t *Y, const float *scale, uint16_t *Yh,
                           void *ws, size_t ws_bytes, void *stream);

nm_status nm_gemm_i8_dense_ex(const int8_t *X, int m, const int8_t *W, int n, int k,
                              int32_t *Y, const float *scale, uint16_t *Yh,
                              void *ws, size_t ws_bytes, void *stream, const nm_plan *plan);

/* ---------------------------------------------------------------- expansion
 * The decode of a compact weight (Sec. 4.2) as a pass of its own: the form a
 * plan with expand = 1 builds in its workspace, written to a caller buffer
 * instead, so that a caller can run it ahead of the GEMM that reads it (on
 * another stream, overlapping earlier work), or once at load time. */

/* Descriptor and size of the expanded form of a compact packed weight (the
 * C14, C18, C28 and MKn layouts):
 *   C14, C18, C28 -> NM_LAYOUT_SP42 (the descriptor nm_compress_size gives for
 *                    2:4 and the same n, k): the values (expanded->vals_bytes)
 *                    followed by the positions (expanded->meta_bytes) in one
 *                    buffer.  Every group holds the layout's nonzeros; the
 *                    padding slots hold zeros, at positions that need not be
 *                    the canonical ones (nm_decompress may reject the result;
 *                    the GEMMs compute with it exactly).
 *   MK3, MK4, MK5 -> NM_LAYOUT_DENSE (the descriptor of 8:8 and the same n, k):
 *                    W [n x k] row-major, meta_bytes 0.
 * *bytes = expanded->vals_bytes + expanded->meta_bytes.  Host only.  Errors:
 * NM_ERR_ARG (NULL pointer, inconsistent desc, or a layout that is already an
 * operand form: SP42 or DENSE). */
nm_status nm_expand_size(const nm_desc *desc, nm_desc *expanded, size_t *bytes);

/* Expands a device packed weight (vals, meta as for nm_spmm) into the device
 * buffer out of out_bytes (>= the size above), on `stream`, asynchronously.
 * The result is a packed weight of the expanded descriptor: nm_spmm_ex (or
 * nm_spmm_out) with that descriptor, vals = out and meta = out +
 * expanded->vals_bytes (NULL for DENSE) computes the same outputs as the
 * compact weight.  Errors: as nm_expand_size, NM_ERR_ARG for a NULL or
 * misaligned pointer, NM_ERR_WORKSPACE when out_bytes is too small (nothing
 * written), NM_ERR_HIP. */
nm_status nm_expand(const nm_desc *desc, const int8_t *vals, const uint8_t *meta, int8_t *out,
                    size_t out_bytes, void *stream);

/* An expansion (nm_expand's work) that a GEMM launch carries along: the
 * compact packed weight (desc, device vals and meta) and the device buffer
 * out of out_bytes (>= nm_expand_size) it is expanded into. */
typedef struct nm_expand_job {
    const nm_desc *desc;
    const int8_t *vals;
    const uint8_t *meta;
    int8_t *out;
    size_t out_bytes;
} nm_expand_job;

/* ---------------------------------------------------------------- INT8 chaining
 * The paper deploys the linears in INT8 end to end (Sec. 6.3).  Between two
 * linears the int32 result must become the next linear's int8 input; the
 * entry points below do that inside the GEMM's epilogue (requantisation) and,
 * for the first linear, on binary16 activations (quantisation).
 *
 * q8(v): the binary32 value v rounded to the nearest integer, ties to even,
 * saturated to [-127, 127]; NaN gives 0.  Products are rounded to binary32
 * before q8, so a code is decided in binary32.  Symmetric per-tensor
 * quantisation of the next input with scale s_y is qscale[j] = s_x * s_w[j] /
 * s_y (per channel because the weight scales are). */

/* Outputs of one GEMM: any non-empty subset.
 *   y       device int32 [m x n]  Y = X W^T
 *   yh      device binary16 [m x n] fp16(fp32(Y) * scale[j]), needs scale
 *   scale   device float32 [n]
 *   yq      device int8 [m x n]  q8(fp32(Y) * qscale[j]), needs qscale
 *   qscale  device float32 [n]
 * Every non-NULL pointer must be 16-byte aligned. */
typedef struct nm_outputs {
    int32_t *y;
    uint16_t *yh;
    const float *scale;
    int8_t *yq;
    const float *qscale;
} nm_outputs;

/* nm_spmm_ex with the outputs given by `out` (host struct, read during the
 * call).  plan may be NULL.  Errors as nm_spmm_ex; NM_ERR_ARG also for
 * out == NULL, no output, or an output without its multiplier array. */
nm_status nm_spmm_out(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                      const nm_desc *desc, const nm_outputs *out,
                      void *ws, size_t ws_bytes, void *stream, const nm_plan *plan);

/* nm_spmm_out without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  A plan that needs a workspace (split_k > 1) uses a
 * scratch array that the library holds in device memory instead: the 16384-byte
 * counter block plus 32 MiB (33570816 bytes in all), one copy per device, kept
 * until the process ends.  The call itself allocates nothing.  The first call
 * on a device looks the array up and clears its counters with a kernel on
 * `stream`; every call leaves them at zero again.  All calls on one device
 * share that array, so calls that may overlap on one device (other streams,
 * other host threads without ordering) race on it and must not be issued.
 * Arguments as nm_spmm_out without ws / ws_bytes; plan may be NULL (the
 * planner's).  Errors as nm_spmm_out; NM_ERR_WORKSPACE when the plan needs
 * more than the array holds (nm_workspace_size() > 33570816), NM_ERR_HIP when
 * the array cannot be looked up. */
nm_status nm_spmm_noalloc(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                          const nm_desc *desc, const nm_outputs *out, void *stream, const nm_plan *plan);

/* nm_gemm_i8_dense_ex with the outputs given by `out`. */
nm_status nm_gemm_i8_dense_out(const int8_t *X, int m, const int8_t *W, int n, int k,
                               const nm_outputs *out,
                               void *ws, size_t ws_bytes, void *stream, const nm_plan *plan);

/* nm_spmm_out (or nm_gemm_i8_dense_out) that also runs `job` in the same
 * kernel launch: workgroups appended after the GEMM's own expand the job's
 * weight, one block per wave, so they are dispatched last and fill the
 * compute units the GEMM's final round of workgroups leaves idle.  A caller
 * that runs linears in sequence expands the next linear's weight this way and
 * then runs that linear on the expanded form (nm_spmm_out with the descriptor
 * nm_expand_size gives, vals = job->out, meta = job->out + its vals_bytes),
 * with no launch of its own for the expansion.  job == NULL is exactly
 * nm_spmm_out.  With m == 0 the job is still run (alone).  Errors: as
 * nm_spmm_out, plus those of nm_expand for the job, and NM_ERR_ARG when
 * job->out overlaps X, the weight, an output, the workspace the plan uses or
 * the job's own packed weight (all checked before anything is launched). */
nm_status nm_spmm_out_expand(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                             const nm_desc *desc, const nm_outputs *out, void *ws, size_t ws_bytes,
                             void *stream, const nm_plan *plan, const nm_expand_job *job);
nm_status nm_gemm_i8_dense_out_expand(const int8_t *X, int m, const int8_t *W, int n, int k,
                                      const nm_outputs *out, void *ws, size_t ws_bytes, void *stream,
                                      const nm_plan *plan, const nm_expand_job *job);

/* Quantisation of binary16 activations: xq[c] = q8(fp32(x[c]) * inv_scale)
 * for 0 <= c < count (a per-tensor scale s_x gives inv_scale = 1 / s_x).
 * x: device binary16 bits, xq: device int8, both 16-byte aligned; count == 0
 * is a no-op (no pointer examined).  Asynchronous on `stream`.  Errors:
 * NM_ERR_SHAPE (count < 0), NM_ERR_ARG (NULL or misaligned pointer),
 * NM_ERR_HIP. */
nm_status nm_quantize_f16(const uint16_t *x, int64_t count, float inv_scale, int8_t *xq, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* NMSPMM_H */
