/*
 * nmsearch.h -- latency predictor and layer-wise N:M search of libnmspmm
 * (paper: "Realizable N:M Sparse Transformer Inference via Search-Kernel
 * Co-Design", Sec. 5).  Host code only, synchronous, no GPU needed; all
 * pointers are host memory owned by the caller.
 *
 * Predictor (Sec. 5.1, Eq. 1).  A lookup table gives the measured latency
 * t_l(s) of layer l's GEMM under sparsity setting s (measured with the GEMM
 * entry points of nmspmm.h).  The end-to-end latency of a configuration
 * s = (s_1 .. s_L) is predicted as
 *     T_pred(s) = sum_l gamma_l * t_l(s_l) + b,     gamma_l >= 0, b >= 0,
 * with (gamma, b) calibrated by non-negative least squares on a few measured
 * full-model latencies.
 *
 * Search (Sec. 5.2, Algorithm 1).  The search space is the N:8 family: layer
 * l runs N_l:8 with N_l in 1..8 (8 = dense).  Within the latency budget it
 * maximises a caller-supplied fitness (the paper's inherited supernet
 * accuracy, Eq. 3) with a (1 + lambda) evolutionary loop whose offspring are
 * made by three stages: overshoot (densify a few random layers past the
 * budget), repair (sparsify random layers until the budget holds again) and
 * refine (densify random layers while that keeps the budget and does not
 * lower the fitness).
 */
#ifndef NMSEARCH_H
#define NMSEARCH_H

#include <stdint.h>

#include "nmspmm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Non-negative least squares: x = argmin ||A x - y||_2 subject to x >= 0
 * (the calibration of Eq. 1), by the Lawson-Hanson active-set method.
 *   A      [rows x cols] row-major
 *   y      [rows]
 *   x      [cols] (output)
 *   rnorm  ||A x - y||_2 (output, may be NULL)
 * A column that is numerically dependent on the columns already in use is
 * left at zero.  Errors: NM_ERR_ARG (NULL pointer, size < 1, non-finite
 * input), NM_ERR_SHAPE (no convergence within 3 * cols + 10 iterations). */
nm_status nm_nnls(const double *A, int rows, int cols, const double *y, double *x, double *rnorm);

/* Calibration of Eq. 1: t is [configs x layers] row-major, row c holding the
 * table latencies t_l(s_l) of measured configuration c, T [configs] its
 * measured end-to-end latency.  Writes gamma [layers] and *b.  Errors as
 * nm_nnls. */
nm_status nm_latency_fit(const double *t, int configs, int layers, const double *T, double *gamma, double *b);

/* T_pred of one configuration (Eq. 1): *T = sum_l gamma[l] * t[l] + b, summed
 * in order of l. */
nm_status nm_latency_predict(const double *t, int layers, const double *gamma, double b, double *T);

/* Fitness of a configuration: n_of_layer[l] in 1..8.  Must not keep the
 * pointer.  A NaN result counts as -infinity. */
typedef double (*nm_fitness_fn)(const int32_t *n_of_layer, int layers, void *user);

typedef struct nm_search_params {
    int32_t generations;   /* G >= 0 */
    int32_t offspring;     /* lambda >= 1 */
    int32_t overshoot;     /* layers densified by the overshoot stage, >= 1 */
    int32_t reserved;      /* must be 0 */
    uint64_t seed;         /* all random draws come from this seed */
} nm_search_params;

/* Algorithm 1 on the predictor.
 *   lut      [layers x 8] row-major: lut[l * 8 + (N - 1)] = t_l(N:8)
 *   gamma, b calibrated predictor (Eq. 1)
 *   target   latency budget T_target (same unit as T_pred)
 *   fitness  accuracy stand-in, called for feasible configurations only
 *   best     [layers] (output): the final configuration, values 1..8
 *   best_fitness (output, may be NULL), trace [generations + 1] (output, may
 *   be NULL): the parent's fitness before each generation and at the end.
 * Random draws: SplitMix64 (Steele, Lea and Flood, 2014) used as a
 * counter-based generator, draw i = mix64(seed + (i + 1) * 0x9E3779B97F4A7C15);
 * an index below n is floor(draw * n / 2^64).  Errors: NM_ERR_ARG (bad
 * argument), NM_ERR_SHAPE (no uniform configuration meets the budget). */
nm_status nm_search(int layers, const double *lut, const double *gamma, double b, double target,
                    nm_fitness_fn fitness, void *user, const nm_search_params *params, int32_t *best,
                    double *best_fitness, double *trace);

#ifdef __cplusplus
}
#endif

#endif /* NMSEARCH_H */
