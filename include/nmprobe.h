/* nmprobe.h -- measurement aid of libnmspmm (not part of the method).
 *
 * The matrix-instruction rate this GPU sustains on given operand values: the
 * practical ceiling beside the data-sheet peak.  Under random int8 operands
 * the chip lowers its clock (power), so a structured-sparse or dense int8
 * matrix instruction stream runs below the peak derived from the nominal
 * clock; the GEMM kernels' compute-bound throughput is compared with this.
 */
#ifndef NMPROBE_H
#define NMPROBE_H

#include <stdint.h>

#include "nmspmm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Operand table of the rate loop: NM_PROBE_WORDS int32 words in device memory.
 *   words [0, 2048):    A operands, 8 fragments x 64 lanes x 4 words
 *   words [2048, 4096): B operands, 4 fragments x 64 lanes x 8 words
 * (the structured-sparse position words are fixed valid patterns). */
#define NM_PROBE_WORDS 4096

/* Launches `workgroups` workgroups of 4 waves; each wave loads its operands
 * from `operands` and issues iters x 8 independent matrix instructions of
 * `kind` (four of the dense ones being the second k-half of the other four,
 * as in the dense GEMM):
 *   NM_KIND_SP42  -- v_smfmac_i32_16x16x128_i8, 2*16*16*128 dense-equivalent
 *                    ops each (half of them on stored zeros)
 *   NM_KIND_DENSE -- v_mfma_i32_16x16x64_i8, 2*16*16*64 ops each
 * and writes one int32 per thread to out[workgroups x 256] (so the loop is
 * not removed).  If `ticks` is not NULL, wave 0 of workgroup w writes
 * ticks[2w] = shader-clock cycles and ticks[2w + 1] = real-time counter
 * ticks spent in its loop (the real-time counter runs at nm_wall_clock_khz),
 * from which the shader clock during the loop follows.  Asynchronous on
 * `stream` (a hipStream_t, NULL = default); time it with events on that
 * stream.  The caller owns the buffers (device memory).
 * Errors: NM_ERR_ARG for a NULL operands/out, another kind, iters < 1 or
 * workgroups < 1; NM_ERR_HIP if the launch fails. */
nm_status nm_probe_mfma_rate(int kind, const int32_t *operands, int iters, int workgroups, int32_t *out,
                             int64_t *ticks, void *stream);

/* Rate of the real-time counter of the current device in kHz (host query).
 * Errors: NM_ERR_ARG for NULL; NM_ERR_HIP if the device query fails. */
nm_status nm_wall_clock_khz(int32_t *khz);

/* One matrix instruction on one wave (64 lanes), operands given per lane, so
 * a test can pin the (lane, register byte) <-> (row, k, column) maps that the
 * packed weight layout and the GEMM kernels rely on.  Device buffers, caller
 * owned, int32 words, lane-major:
 *   kind NM_KIND_SP42 (v_smfmac_i32_16x16x128_i8):
 *     a[64 x 4] (16 value bytes per lane), b[64 x 8] (32 bytes per lane),
 *     pos[64] (one position word per lane), d[64 x 4]
 *   kind NM_KIND_DENSE (v_mfma_i32_16x16x64_i8):
 *     a[64 x 4], b[64 x 4], pos unused (may be NULL), d[64 x 4]
 * d receives the lane's four accumulator words of D = A x B (C = 0).
 * Asynchronous on `stream`.  Errors: NM_ERR_ARG for a NULL buffer or another
 * kind; NM_ERR_HIP if the launch fails. */
nm_status nm_probe_mfma_layout(int kind, const int32_t *a, const int32_t *b, const int32_t *pos, int32_t *d,
                               void *stream);

/* The output stream of a GEMM plan alone: launches the plan's kernel for an
 * [m x n] output with the reduction skipped (no operand loads, no matrix
 * instructions), so every output element is written with the value of an
 * empty sum (int32 0; fp16 and int8 of 0 times the scale, 0 for finite
 * scales) through the same epilogue, store pattern and cache policy as
 * nm_spmm_out.  Timing it beside the real call
 * gives the ceiling the GEMM's own stores set.  plan: a plan of an
 * output-split tile layout (the layouts nm_tile_info reports for k_gemm) with
 * split_k == 1, for the plan's kind; out: as for nm_spmm_out (device buffers,
 * caller owned; scales are read).  Asynchronous on `stream`.
 * Errors: NM_ERR_ARG for a NULL plan/out, no output, a missing scale,
 * misaligned pointers, another tile layout or split_k != 1; NM_ERR_SHAPE for
 * m < 0, n < 4, n % 4 != 0 or m * n >= 2^29; NM_ERR_HIP if the launch fails.
 * m == 0 writes nothing. */
nm_status nm_probe_store_only(const nm_plan *plan, int m, int n, const nm_outputs *out, void *stream);

/* Timing events (hipEvent_t behind a void pointer) created with
 * hipEventDisableSystemFence: recording one adds no system-scope memory
 * fence (no cache write-back and invalidation) when it completes, so events
 * placed between the GEMMs of a sequence time them without changing what the
 * caches hold or adding that fence's cost to the next GEMM.  Only for timing:
 * elapsed times are valid once the host has synchronised with the stream.
 *   nm_probe_event_create:      *event = a new event (caller destroys it)
 *   nm_probe_event_destroy:     frees it
 *   nm_probe_event_record:      records it on `stream` (a hipStream_t, NULL =
 *                               default), asynchronously
 *   nm_probe_event_elapsed_ms:  *ms = time from `start` to `stop`, both
 *                               recorded and complete
 * Errors: NM_ERR_ARG for a NULL pointer; NM_ERR_HIP if the runtime call fails
 * (e.g. an event not yet complete). */
nm_status nm_probe_event_create(void **event);
nm_status nm_probe_event_destroy(void *event);
nm_status nm_probe_event_record(void *event, void *stream);
nm_status nm_probe_event_elapsed_ms(float *ms, void *start, void *stop);

#ifdef __cplusplus
}
#endif

#endif /* NMPROBE_H */
