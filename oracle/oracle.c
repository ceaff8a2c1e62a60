/*
 * oracle.c -- plain, slow CPU definition of the N:M sparse INT8 GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header, table or helper with the
 * HIP library; the two meet only at plain arrays produced by the seeded input
 * generators.
 *
 * What is computed (paper: "Realizable N:M Sparse Transformer Inference via
 * Search-Kernel Co-Design"):
 *   - N:M semi-structured sparsity (Sec. 2.1): every aligned group of M
 *     consecutive weights along the reduction axis keeps at most N nonzeros.
 *   - The packed form B_pack (Sec. 4.2): for each window, the kept values
 *     together with their positions inside the window.
 *   - The sparse product (Sec. 4.2, Micro-Dense): the output is the plain
 *     product of the activations with the sparse weights; the packed form only
 *     changes how it is evaluated.  Y[i][j] = sum_t X[i][t] * W[j][t], with
 *     W [n x k] row-major (groups along k) and X [m x k] row-major.
 *   - The optional per-output-channel dequantisation to fp16 (an epilogue the
 *     paper's INT8 deployment implies, Sec. 6.3): Yh = fp16(Y * scale[j]).
 *
 * Arithmetic: exact integers (int64 accumulation, checked to fit int32) and
 * one rounding from double to IEEE binary16 (nearest, ties to even).  No
 * blocking, no SIMD, no reordering: each function is the definition written
 * out so that it can be checked against the paper by eye.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#include <pthread.h>
#include <unistd.h>

#define ORC_OK 0
#define ORC_ERR_ARG 1
#define ORC_ERR_OVERFLOW 2
#define ORC_ERR_PATTERN 3

/* ---- N:M validity (Sec. 2.1) -------------------------------------------
 * Returns ORC_OK when every aligned window [g*M, g*M+M) of every row of W
 * holds at most N nonzeros.  On the first violation (row-major order) returns
 * ORC_ERR_PATTERN and reports the row and window index. */
int orc_nm_check(const int8_t *W, int n, int k, int N, int M, int *bad_row, int *bad_group)
{
    if (!W || n < 0 || k < 0 || M <= 0 || N < 0 || N > M || k % M != 0) return ORC_ERR_ARG;
    for (int j = 0; j < n; ++j) {
        for (int g = 0; g < k / M; ++g) {
            int nnz = 0;
            for (int p = 0; p < M; ++p)
                if (W[(int64_t)j * k + g * M + p] != 0) nnz++;
            if (nnz > N) {
                if (bad_row) *bad_row = j;
                if (bad_group) *bad_group = g;
                return ORC_ERR_PATTERN;
            }
        }
    }
    return ORC_OK;
}

/* ---- canonical B_pack, logical form (Sec. 4.2) --------------------------
 * For each row j and window g there are N slots (value, position-in-window).
 * Slots hold the window's nonzeros in ascending position; the remaining slots
 * are padding: value 0 at the smallest positions not already used, so the N
 * positions of a window are distinct and ascending.
 * vals and offs are [n][k/M][N]. */
int orc_pack_logical(const int8_t *W, int n, int k, int N, int M, int8_t *vals, uint8_t *offs)
{
    if (!W || !vals || !offs || M <= 0 || N <= 0 || N > M || k % M != 0) return ORC_ERR_ARG;
    int G = k / M;
    for (int j = 0; j < n; ++j) {
        for (int g = 0; g < G; ++g) {
            const int8_t *win = W + (int64_t)j * k + g * M;
            int used[64] = {0};
            int nnz = 0;
            for (int p = 0; p < M; ++p)
                if (win[p] != 0) nnz++;
            if (nnz > N) return ORC_ERR_PATTERN;
            /* positions of the slots: the nonzeros, then the smallest free ones */
            int pos[64];
            int c = 0;
            for (int p = 0; p < M; ++p)
                if (win[p] != 0) { pos[c++] = p; used[p] = 1; }
            for (int p = 0; p < M && c < N; ++p)
                if (!used[p]) { pos[c++] = p; used[p] = 1; }
            /* ascending order of positions (insertion sort, N is tiny) */
            for (int a = 1; a < N; ++a) {
                int v = pos[a], b = a - 1;
                while (b >= 0 && pos[b] > v) { pos[b + 1] = pos[b]; b--; }
                pos[b + 1] = v;
            }
            for (int s = 0; s < N; ++s) {
                int64_t o = ((int64_t)j * G + g) * N + s;
                offs[o] = (uint8_t)pos[s];
                vals[o] = win[pos[s]];
            }
        }
    }
    return ORC_OK;
}

/* Inverse of the logical packing: W[j][g*M + offs] = vals, zero elsewhere. */
int orc_unpack_logical(const int8_t *vals, const uint8_t *offs, int n, int k, int N, int M, int8_t *W)
{
    if (!vals || !offs || !W || M <= 0 || N <= 0 || N > M || k % M != 0) return ORC_ERR_ARG;
    int G = k / M;
    memset(W, 0, (size_t)n * (size_t)k);
    for (int j = 0; j < n; ++j)
        for (int g = 0; g < G; ++g)
            for (int s = 0; s < N; ++s) {
                int64_t o = ((int64_t)j * G + g) * N + s;
                if (offs[o] >= M) return ORC_ERR_ARG;
                W[(int64_t)j * k + g * M + offs[o]] = vals[o];
            }
    return ORC_OK;
}

/* ---- threads: rows of the output are split in contiguous blocks ---------
 * Used only so the oracle can be timed on all host cores; every output value
 * is computed by the same scalar loop whatever the thread count. */
typedef struct {
    const int8_t *X, *W, *vals;
    const uint8_t *offs;
    int m, n, k, N, M;
    int row0, row1;
    int32_t *Y;
    int err;
} orc_job;

static int orc_nthreads(int requested)
{
    if (requested > 0) return requested;
    long c = sysconf(_SC_NPROCESSORS_ONLN);
    return c > 0 ? (int)c : 1;
}

static void *orc_dense_rows(void *arg)
{
    orc_job *J = (orc_job *)arg;
    for (int i = J->row0; i < J->row1; ++i) {
        for (int j = 0; j < J->n; ++j) {
            int64_t acc = 0;
            for (int t = 0; t < J->k; ++t)
                acc += (int64_t)J->X[(int64_t)i * J->k + t] * (int64_t)J->W[(int64_t)j * J->k + t];
            if (acc > INT32_MAX || acc < INT32_MIN) { J->err = ORC_ERR_OVERFLOW; acc = 0; }
            J->Y[(int64_t)i * J->n + j] = (int32_t)acc;
        }
    }
    return NULL;
}

static void *orc_packed_rows(void *arg)
{
    orc_job *J = (orc_job *)arg;
    int G = J->k / J->M;
    for (int i = J->row0; i < J->row1; ++i) {
        for (int j = 0; j < J->n; ++j) {
            int64_t acc = 0;
            for (int g = 0; g < G; ++g)
                for (int s = 0; s < J->N; ++s) {
                    int64_t o = ((int64_t)j * G + g) * J->N + s;
                    acc += (int64_t)J->vals[o] * (int64_t)J->X[(int64_t)i * J->k + g * J->M + J->offs[o]];
                }
            if (acc > INT32_MAX || acc < INT32_MIN) { J->err = ORC_ERR_OVERFLOW; acc = 0; }
            J->Y[(int64_t)i * J->n + j] = (int32_t)acc;
        }
    }
    return NULL;
}

static int orc_run_rows(orc_job proto, int nthreads, void *(*fn)(void *))
{
    int T = orc_nthreads(nthreads);
    if (T > proto.m) T = proto.m > 0 ? proto.m : 1;
    orc_job *jobs = (orc_job *)calloc((size_t)T, sizeof(orc_job));
    pthread_t *th = (pthread_t *)calloc((size_t)T, sizeof(pthread_t));
    if (!jobs || !th) { free(jobs); free(th); return ORC_ERR_ARG; }
    for (int t = 0; t < T; ++t) {
        jobs[t] = proto;
        jobs[t].row0 = (int)((int64_t)proto.m * t / T);
        jobs[t].row1 = (int)((int64_t)proto.m * (t + 1) / T);
        jobs[t].err = ORC_OK;
    }
    for (int t = 1; t < T; ++t) pthread_create(&th[t], NULL, fn, &jobs[t]);
    fn(&jobs[0]);
    for (int t = 1; t < T; ++t) pthread_join(th[t], NULL);
    int err = ORC_OK;
    for (int t = 0; t < T; ++t)
        if (jobs[t].err) err = jobs[t].err;
    free(jobs);
    free(th);
    return err;
}

/* ---- the plain product Y = X * W^T ---------------------------------------
 * X int8 [m x k], W int8 [n x k] (already decompressed), Y int32 [m x n].
 * Exact int64 accumulation; ORC_ERR_OVERFLOW if a value leaves int32. */
int orc_matmul_i8(const int8_t *X, const int8_t *W, int m, int n, int k, int32_t *Y, int nthreads)
{
    if (!X || !W || !Y || m < 0 || n < 0 || k < 0) return ORC_ERR_ARG;
    if (m == 0 || n == 0) return ORC_OK;
    orc_job J;
    memset(&J, 0, sizeof J);
    J.X = X; J.W = W; J.m = m; J.n = n; J.k = k; J.Y = Y;
    return orc_run_rows(J, nthreads, orc_dense_rows);
}

/* Same definition at a list of (row, col) positions only. */
int orc_matmul_i8_sampled(const int8_t *X, const int8_t *W, int m, int n, int k,
                          const int64_t *rows, const int64_t *cols, int64_t count, int32_t *out)
{
    if (!X || !W || !rows || !cols || !out || k < 0) return ORC_ERR_ARG;
    int err = ORC_OK;
    for (int64_t c = 0; c < count; ++c) {
        int64_t i = rows[c], j = cols[c];
        if (i < 0 || i >= m || j < 0 || j >= n) return ORC_ERR_ARG;
        int64_t acc = 0;
        for (int t = 0; t < k; ++t)
            acc += (int64_t)X[i * k + t] * (int64_t)W[j * k + t];
        if (acc > INT32_MAX || acc < INT32_MIN) { err = ORC_ERR_OVERFLOW; acc = 0; }
        out[c] = (int32_t)acc;
    }
    return err;
}

/* ---- the product evaluated from the packed form (Sec. 4.2) ---------------
 * Y[i][j] = sum over windows g and slots s of
 *           vals[j][g][s] * X[i][g*M + offs[j][g][s]],
 * i.e. each window's kept values meet the activations at their recorded
 * positions.  Equal to orc_matmul_i8 on the unpacked weights. */
int orc_spmm_packed(const int8_t *X, int m, const int8_t *vals, const uint8_t *offs,
                    int n, int k, int N, int M, int32_t *Y, int nthreads)
{
    if (!X || !vals || !offs || !Y || M <= 0 || N <= 0 || N > M || k % M != 0) return ORC_ERR_ARG;
    if (m == 0 || n == 0) return ORC_OK;
    orc_job J;
    memset(&J, 0, sizeof J);
    J.X = X; J.vals = vals; J.offs = offs; J.m = m; J.n = n; J.k = k; J.N = N; J.M = M; J.Y = Y;
    return orc_run_rows(J, nthreads, orc_packed_rows);
}

/* ---- IEEE 754 binary16 from double, round to nearest, ties to even -------
 * binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Normal values have spacing 2^(e-10) in the binade [2^e, 2^(e+1)),
 * e in [-14, 15]; below 2^-14 the spacing is 2^-24 (subnormals).  The value is
 * divided by its spacing (a power of two, so exactly), rounded to an integer
 * with ties to even, and the integer is turned back into fields. */
uint16_t orc_f64_to_f16(double x)
{
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x)) return (uint16_t)(sign | 0x7E00u);
    double a = fabs(x);
    if (isinf(a)) return (uint16_t)(sign | 0x7C00u);
    if (a == 0.0) return sign;
    int e2;
    double spacing;
    int normal;
    if (a >= ldexp(1.0, -14)) {
        int E;
        (void)frexp(a, &E);      /* a = f * 2^E, f in [0.5, 1): binade exponent is E-1 */
        e2 = E - 1;
        if (e2 > 15) return (uint16_t)(sign | 0x7C00u);
        spacing = ldexp(1.0, e2 - 10);
        normal = 1;
    } else {
        e2 = -14;
        spacing = ldexp(1.0, -24);
        normal = 0;
    }
    double r = a / spacing;     /* exact: division by a power of two, r < 2^11 */
    double fl = floor(r);
    double frac = r - fl;       /* exact */
    double q = fl;
    if (frac > 0.5) q = fl + 1.0;
    else if (frac == 0.5) q = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
    uint32_t Nq = (uint32_t)q;
    uint32_t bits;
    if (normal) {
        /* Nq in [1024, 2048]; 2048 carries into the next binade */
        bits = ((uint32_t)(e2 + 15) << 10) + (Nq - 1024u);
    } else {
        /* Nq in [0, 1024]; 1024 is exactly the smallest normal 0x0400 */
        bits = Nq;
    }
    if (bits >= 0x7C00u) bits = 0x7C00u;
    return (uint16_t)(sign | bits);
}

void orc_f64_to_f16_array(const double *x, int64_t count, uint16_t *out)
{
    for (int64_t c = 0; c < count; ++c) out[c] = orc_f64_to_f16(x[c]);
}

/* ---- dequantisation epilogue ----------------------------------------------
 * Yh[i][j] = binary16( (double)Y[i][j] * (double)scale[j] ), one rounding. */
int orc_dequant_f16(const int32_t *Y, const float *scale, int m, int n, uint16_t *Yh)
{
    if (!Y || !scale || !Yh || m < 0 || n < 0) return ORC_ERR_ARG;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j)
            Yh[i * n + j] = orc_f64_to_f16((double)Y[i * n + j] * (double)scale[j]);
    return ORC_OK;
}

/* ---- int8 quantisation on either side of a linear ------------------------
 * The paper deploys the linears in INT8 end to end (Sec. 6.3) without
 * spelling out the quantiser.  Reading used here: symmetric and saturating to
 * [-127, 127]; the scale is a binary32 multiplier; the product is rounded to
 * the nearest integer, ties to even, in binary32; NaN quantises to 0.  The
 * code of a value is decided in binary32 because that is the precision the
 * GPU kernels use, so both sides take the same decision. */
static int8_t orc_q8_of(float v)
{
    if (isnan(v)) return 0;
    float r = nearbyintf(v);   /* default rounding mode: nearest, ties to even */
    if (r > 127.0f) r = 127.0f;
    if (r < -127.0f) r = -127.0f;
    return (int8_t)r;
}

/* binary16 bit pattern -> binary32 value (exact): sign, 5-bit exponent with
 * bias 15, 10-bit fraction; exponent 0 holds subnormals f * 2^-24, exponent 31
 * holds infinities (f = 0) and NaNs. */
float orc_f16_to_f32(uint16_t h)
{
    int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
    float mag;
    if (e == 31) mag = f ? NAN : INFINITY;
    else if (e == 0) mag = ldexpf((float)f, -24);
    else mag = ldexpf((float)(f + 1024), e - 25);   /* (1 + f/1024) * 2^(e-15) */
    return s ? -mag : mag;
}

/* Activation quantisation (prologue of the first linear):
 * xq[c] = q8( f32(x[c]) * inv_scale ), x given as binary16 bit patterns. */
int orc_quantize_f16(const uint16_t *x, int64_t count, float inv_scale, int8_t *xq)
{
    if ((!x || !xq) && count > 0) return ORC_ERR_ARG;
    for (int64_t c = 0; c < count; ++c) {
        float v = orc_f16_to_f32(x[c]) * inv_scale;
        xq[c] = orc_q8_of(v);
    }
    return ORC_OK;
}

/* Requantisation epilogue (int32 accumulator -> int8 input of the next
 * linear): Yq[i][j] = q8( f32(Y[i][j]) * qscale[j] ).  f32(Y) rounds to
 * nearest-even when |Y| > 2^24.  A per-tensor requantisation is the case of
 * equal qscale entries; with per-channel weight scales the multiplier
 * s_x * s_w[j] / s_y is per channel anyway. */
int orc_requant_i8(const int32_t *Y, const float *qscale, int m, int n, int8_t *Yq)
{
    if (!Y || !qscale || !Yq || m < 0 || n < 0) return ORC_ERR_ARG;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) {
            float v = (float)Y[i * n + j] * qscale[j];
            Yq[i * n + j] = orc_q8_of(v);
        }
    return ORC_OK;
}
