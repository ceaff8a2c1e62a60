// Host-side stress of the library's CPU code (packing, planner, Eq. 1
// calibration, Algorithm 1) for an AddressSanitizer / UndefinedBehaviorSanitizer
// build: random valid and invalid inputs through every host entry point, with
// the round trips and invariants checked.  Exits non-zero on the first failure
// (the sanitizers abort on their own).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "nmsearch.h"
#include "nmspmm.h"

namespace nmspmm {
nm_status make_plan(int kind, int m, int n, int k, int out_mode, nm_plan *plan);
nm_status complete_plan(int kind, int m, int n, int k, nm_plan *plan);
}

#define CHECK(c)                                                      \
    do {                                                              \
        if (!(c)) {                                                   \
            std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            std::exit(1);                                             \
        }                                                             \
    } while (0)

static std::mt19937_64 rng(20260);
static int uni(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }

// W [n x k] with at most N nonzeros in every aligned window of M (random count and places).
static std::vector<int8_t> nm_weight(int n, int k, int N, int M) {
    std::vector<int8_t> W((size_t)n * k, 0);
    for (int r = 0; r < n; ++r)
        for (int w = 0; w < k / M; ++w) {
            int cnt = uni(0, N);
            std::vector<int> pos(M);
            for (int i = 0; i < M; ++i) pos[i] = i;
            std::shuffle(pos.begin(), pos.end(), rng);
            for (int i = 0; i < cnt; ++i) {
                int v = uni(-128, 127);
                W[(size_t)r * k + w * M + pos[i]] = (int8_t)(v == 0 ? 1 : v);
            }
        }
    return W;
}

static void pack_round_trips() {
    for (int M : {4, 8})
        for (int N = 1; N <= M; ++N)
            for (int rep = 0; rep < 6; ++rep) {
                const int n = 4 * uni(1, 20), k = 16 * uni(1, 24);
                if (k % M) continue;
                nm_desc d;
                CHECK(nm_compress_size(n, k, N, M, &d) == NM_OK);
                std::vector<int8_t> W = nm_weight(n, k, N, M), back((size_t)n * k, 7);
                std::vector<int8_t> vals((size_t)d.vals_bytes);
                std::vector<uint8_t> meta((size_t)d.meta_bytes);
                CHECK(nm_compress(W.data(), n, k, N, M, vals.data(), meta.data(), &d) == NM_OK);
                CHECK(nm_decompress(&d, vals.data(), meta.data(), back.data()) == NM_OK);
                CHECK(std::memcmp(W.data(), back.data(), W.size()) == 0);
                if (N < M) {
                    // one window over the limit is rejected and named
                    const int r = uni(0, n - 1), w = uni(0, k / M - 1);
                    for (int i = 0; i < M; ++i) W[(size_t)r * k + w * M + i] = (int8_t)(i + 1);
                    CHECK(nm_compress(W.data(), n, k, N, M, vals.data(), meta.data(), &d) == NM_ERR_PATTERN);
                    CHECK(d.bad_row >= 0 && d.bad_row <= r && d.bad_group >= 0);
                }
            }
    nm_desc d;
    CHECK(nm_compress_size(64, 100, 2, 4, &d) == NM_ERR_SHAPE);   // k % 16
    CHECK(nm_compress_size(6, 128, 2, 4, &d) == NM_ERR_SHAPE);    // n % 4
    CHECK(nm_compress_size(64, 128, 3, 5, &d) == NM_ERR_UNSUPPORTED);
    CHECK(nm_compress_size(64, 128, 2, 4, nullptr) == NM_ERR_ARG);
    CHECK(nm_compress(nullptr, 64, 128, 2, 4, nullptr, nullptr, &d) == NM_ERR_ARG);
}

static void planner() {
    for (int kind = NM_KIND_SP42; kind <= NM_KIND_MK5; ++kind)
        for (int rep = 0; rep < 400; ++rep) {
            const int m = rep % 7 == 0 ? 0 : uni(1, 200000), n = 4 * uni(1, 4096), ks = uni(1, 64);
            nm_plan p;
            const nm_status s = nmspmm::make_plan(kind, m, n, 128 * ks, NM_OUT_I32 | NM_OUT_F16, &p);
            CHECK(s == NM_OK || s == NM_ERR_SHAPE);
            if (s != NM_OK) continue;
            CHECK(p.split_k == 1 && p.grid >= 1 && p.tile_n >= 16 && p.tile_m >= 16);
            for (int t = -1; t < 32; ++t)  // past both ends of the tile table too
                for (int split : {1, 2, 4, 8, 3}) {
                    nm_plan q;
                    q.kind = kind;
                    q.tile = t;
                    q.split_k = split;
                    q.expand = (t & 1) && kind != NM_KIND_SP42 && kind != NM_KIND_DENSE;
                    const nm_status c = nmspmm::complete_plan(kind, m, n, 128 * ks, &q);
                    CHECK(c == NM_OK || c == NM_ERR_ARG || c == NM_ERR_SHAPE);
                    if (split == 3) CHECK(c == NM_ERR_ARG);
                }
        }
}

static void latency_model() {
    for (int rep = 0; rep < 200; ++rep) {
        const int rows = uni(1, 40), cols = uni(1, 14);
        std::vector<double> A((size_t)rows * cols), y(rows), x(cols, -1.0);
        for (double &a : A) a = std::uniform_real_distribution<double>(0.0, 5.0)(rng);
        for (double &v : y) v = std::uniform_real_distribution<double>(-1.0, 10.0)(rng);
        double rn = -1.0;
        const nm_status s = nm_nnls(A.data(), rows, cols, y.data(), x.data(), &rn);
        CHECK(s == NM_OK || s == NM_ERR_SHAPE);
        if (s == NM_OK) {
            for (double v : x) CHECK(v >= 0.0 && std::isfinite(v));
            CHECK(rn >= 0.0);
        }
    }
    const int layers = 12, configs = 30;
    std::vector<double> t((size_t)configs * layers), T(configs), g(layers);
    for (int c = 0; c < configs; ++c) {
        T[c] = 3.0;
        for (int l = 0; l < layers; ++l) {
            t[(size_t)c * layers + l] = std::uniform_real_distribution<double>(1.0, 9.0)(rng);
            T[c] += (1.0 + 0.1 * l) * t[(size_t)c * layers + l];
        }
    }
    double b = -1.0, Tp = 0.0;
    CHECK(nm_latency_fit(t.data(), configs, layers, T.data(), g.data(), &b) == NM_OK);
    CHECK(nm_latency_predict(t.data(), layers, g.data(), b, &Tp) == NM_OK);
    CHECK(std::fabs(Tp - T[0]) < 1e-6 * T[0]);
    CHECK(nm_nnls(nullptr, 1, 1, T.data(), g.data(), nullptr) == NM_ERR_ARG);
}

static double fitness(const int32_t *n_of_layer, int layers, void *) {
    double f = 0.0;
    for (int l = 0; l < layers; ++l) f += std::log((double)n_of_layer[l]);
    return f;
}

static void search() {
    for (int rep = 0; rep < 20; ++rep) {
        const int layers = uni(1, 40);
        std::vector<double> lut((size_t)layers * 8), gamma(layers, 1.0);
        for (int l = 0; l < layers; ++l)
            for (int N = 1; N <= 8; ++N) lut[(size_t)l * 8 + N - 1] = 1.0 + N * (0.5 + 0.1 * uni(0, 5));
        double dense = 0.0, sparse = 0.0;
        for (int l = 0; l < layers; ++l) dense += lut[(size_t)l * 8 + 7], sparse += lut[(size_t)l * 8];
        const double target = sparse + (dense - sparse) * std::uniform_real_distribution<double>(0.0, 1.0)(rng);
        nm_search_params p{uni(0, 12), uni(1, 6), uni(1, 5), 0, (uint64_t)rep};
        std::vector<int32_t> best(layers);
        std::vector<double> trace((size_t)p.generations + 1);
        double bf = 0.0;
        const nm_status s = nm_search(layers, lut.data(), gamma.data(), 0.0, target, fitness, nullptr, &p,
                                      best.data(), &bf, trace.data());
        CHECK(s == NM_OK || s == NM_ERR_SHAPE);
        if (s == NM_OK) {
            double T = 0.0;
            for (int l = 0; l < layers; ++l) {
                CHECK(best[l] >= 1 && best[l] <= 8);
                T += lut[(size_t)l * 8 + best[l] - 1];
            }
            CHECK(T <= target * (1 + 1e-12));
            for (int g = 1; g <= p.generations; ++g) CHECK(trace[g] >= trace[g - 1]);
        }
    }
}

int main() {
    pack_round_trips();
    planner();
    latency_model();
    search();
    std::printf("host driver: all checks passed\n");
    return 0;
}
