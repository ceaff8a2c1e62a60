// LUT latency predictor of the layer-wise search (paper Sec. 5.1, Eq. 1):
// T_pred = sum_l gamma_l * t_l(s_l) + b with gamma_l, b >= 0 calibrated by
// non-negative least squares on a few full-model measurements.  Host only.
//
// NNLS is the active-set method of Lawson and Hanson ("Solving Least Squares
// Problems", 1974, ch. 23): grow a passive set P from the variable of largest
// positive gradient, solve unconstrained least squares on P (Householder QR),
// and when that solution leaves the feasible region step back to its boundary
// and return the variables that reached zero to the active set.
#include <cmath>
#include <cstdint>
#include <vector>

#include "nmsearch.h"

namespace {

// min ||A[:, P] s - y||_2 by Householder QR of the columns in P (A row-major
// rows x cols).  Returns false when a column of P is numerically dependent on
// the ones before it (then `bad` is its position in P).
bool least_squares(const double *A, int rows, int cols, const std::vector<int> &P, const double *y, double tol,
                   std::vector<double> &s, int *bad) {
    const int p = (int)P.size();
    std::vector<double> R((size_t)rows * p);  // column-major copy of A[:, P]
    for (int c = 0; c < p; ++c)
        for (int i = 0; i < rows; ++i) R[(size_t)c * rows + i] = A[(size_t)i * cols + P[c]];
    std::vector<double> r(y, y + rows);
    std::vector<double> v(rows);
    for (int j = 0; j < p; ++j) {
        double *col = &R[(size_t)j * rows];
        double norm = 0.0;
        for (int i = j; i < rows; ++i) norm += col[i] * col[i];
        norm = std::sqrt(norm);
        if (j >= rows || norm <= tol) {
            *bad = j;
            return false;
        }
        const double alpha = col[j] > 0 ? -norm : norm;
        double vv = 0.0;
        for (int i = j; i < rows; ++i) {
            v[i] = col[i] - (i == j ? alpha : 0.0);
            vv += v[i] * v[i];
        }
        // apply H = I - 2 v v^T / (v^T v) to the remaining columns and to r
        for (int c = j; c < p; ++c) {
            double *cc = &R[(size_t)c * rows];
            double d = 0.0;
            for (int i = j; i < rows; ++i) d += v[i] * cc[i];
            const double f = 2.0 * d / vv;
            for (int i = j; i < rows; ++i) cc[i] -= f * v[i];
        }
        double d = 0.0;
        for (int i = j; i < rows; ++i) d += v[i] * r[i];
        const double f = 2.0 * d / vv;
        for (int i = j; i < rows; ++i) r[i] -= f * v[i];
    }
    s.assign(p, 0.0);
    for (int j = p - 1; j >= 0; --j) {
        double acc = r[j];
        for (int c = j + 1; c < p; ++c) acc -= R[(size_t)c * rows + j] * s[c];
        s[j] = acc / R[(size_t)j * rows + j];
    }
    return true;
}

}  // namespace

extern "C" nm_status nm_nnls(const double *A, int rows, int cols, const double *y, double *x, double *rnorm) {
    if (!A || !y || !x || rows < 1 || cols < 1) return NM_ERR_ARG;
    double anorm = 0.0;
    for (int64_t i = 0; i < (int64_t)rows * cols; ++i) {
        if (!std::isfinite(A[i])) return NM_ERR_ARG;
        anorm = std::fmax(anorm, std::fabs(A[i]));
    }
    for (int i = 0; i < rows; ++i)
        if (!std::isfinite(y[i])) return NM_ERR_ARG;
    const double eps = 2.220446049250313e-16;
    const double tol = 10.0 * eps * anorm * (rows > cols ? rows : cols);

    std::vector<double> xv(cols, 0.0), w(cols), resid(rows), s;
    std::vector<char> in_p(cols, 0), excluded(cols, 0);
    auto gradient = [&]() {
        for (int i = 0; i < rows; ++i) {
            double acc = y[i];
            for (int c = 0; c < cols; ++c) acc -= A[(size_t)i * cols + c] * xv[c];
            resid[i] = acc;
        }
        for (int c = 0; c < cols; ++c) {
            double acc = 0.0;
            for (int i = 0; i < rows; ++i) acc += A[(size_t)i * cols + c] * resid[i];
            w[c] = acc;
        }
    };
    const int max_iter = 3 * cols + 10;
    int iter = 0;
    gradient();
    for (;;) {
        // the active variable of largest positive gradient enters P
        int t = -1;
        double best = tol;
        for (int c = 0; c < cols; ++c)
            if (!in_p[c] && !excluded[c] && w[c] > best) best = w[c], t = c;
        if (t < 0) break;
        in_p[t] = 1;
        for (;;) {
            if (++iter > max_iter) return NM_ERR_SHAPE;
            std::vector<int> P;
            for (int c = 0; c < cols; ++c)
                if (in_p[c]) P.push_back(c);
            int bad = -1;
            if (!least_squares(A, rows, cols, P, y, tol, s, &bad)) {
                // a numerically dependent column cannot improve the fit: drop it for good
                in_p[P[bad]] = 0;
                excluded[P[bad]] = 1;
                if (P[bad] == t) break;
                continue;
            }
            bool feasible = true;
            for (size_t j = 0; j < P.size(); ++j) feasible &= s[j] > 0.0;
            if (feasible) {
                for (size_t j = 0; j < P.size(); ++j) xv[P[j]] = s[j];
                break;
            }
            // step from x towards s up to the first variable reaching zero
            double alpha = 1.0;
            for (size_t j = 0; j < P.size(); ++j)
                if (s[j] <= 0.0) {
                    const double a = xv[P[j]] / (xv[P[j]] - s[j]);
                    if (a < alpha) alpha = a;
                }
            for (size_t j = 0; j < P.size(); ++j) {
                xv[P[j]] += alpha * (s[j] - xv[P[j]]);
                if (xv[P[j]] <= tol) {
                    xv[P[j]] = 0.0;
                    in_p[P[j]] = 0;
                }
            }
        }
        gradient();
    }
    double rr = 0.0;
    gradient();
    for (int i = 0; i < rows; ++i) rr += resid[i] * resid[i];
    for (int c = 0; c < cols; ++c) x[c] = xv[c];
    if (rnorm) *rnorm = std::sqrt(rr);
    return NM_OK;
}

extern "C" nm_status nm_latency_fit(const double *t, int configs, int layers, const double *T, double *gamma,
                                    double *b) {
    if (!t || !T || !gamma || !b || configs < 1 || layers < 1) return NM_ERR_ARG;
    const int cols = layers + 1;
    std::vector<double> A((size_t)configs * cols);
    for (int c = 0; c < configs; ++c) {
        for (int l = 0; l < layers; ++l) A[(size_t)c * cols + l] = t[(size_t)c * layers + l];
        A[(size_t)c * cols + layers] = 1.0;
    }
    std::vector<double> x(cols);
    const nm_status st = nm_nnls(A.data(), configs, cols, T, x.data(), nullptr);
    if (st != NM_OK) return st;
    for (int l = 0; l < layers; ++l) gamma[l] = x[l];
    *b = x[layers];
    return NM_OK;
}

extern "C" nm_status nm_latency_predict(const double *t, int layers, const double *gamma, double b, double *T) {
    if (!t || !gamma || !T || layers < 0) return NM_ERR_ARG;
    double total = 0.0;
    for (int l = 0; l < layers; ++l) total += gamma[l] * t[l];
    *T = total + b;
    return NM_OK;
}
