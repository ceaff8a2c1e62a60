// Layer-wise N:M search on the latency predictor (paper Sec. 5.2, Algorithm 1).
// Host only.  The search space is N:8 with N in 1..8 per layer; feasibility is
// T_pred <= target (Eq. 1); the fitness of an infeasible configuration is
// -infinity (Eq. 3), of a feasible one the caller's callback.
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "nmsearch.h"

namespace {

constexpr int kLevels = 8;  // N:8, N = 1..8

// SplitMix64 output function (Steele, Lea, Flood 2014) applied to a counter:
// draw i of a seed is mix(seed + (i + 1) * golden gamma).
struct CounterRng {
    uint64_t seed, next = 0;
    uint64_t draw() {
        uint64_t z = seed + (next + 1) * 0x9E3779B97F4A7C15ull;
        ++next;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    // an index below n: floor(draw * n / 2^64)
    int below(int n) { return (int)(((unsigned __int128)draw() * (unsigned)n) >> 64); }
};

struct Search {
    int L;
    const double *lut, *gamma;
    double b, target;
    nm_fitness_fn fit;
    void *user;
    CounterRng rng;

    double latency(const std::vector<int32_t> &y) const {
        double total = 0.0;
        for (int l = 0; l < L; ++l) total += gamma[l] * lut[(size_t)l * kLevels + (y[l] - 1)];
        return total + b;
    }
    bool feasible(const std::vector<int32_t> &y) const { return latency(y) <= target; }
    double accuracy(const std::vector<int32_t> &y) const {
        const double v = fit(y.data(), L, user);
        return std::isnan(v) ? -std::numeric_limits<double>::infinity() : v;
    }
    double fitness(const std::vector<int32_t> &y) const {
        return feasible(y) ? accuracy(y) : -std::numeric_limits<double>::infinity();
    }

    // Initialisation: the uniform configurations that meet the budget; the
    // fittest (first in N order on ties).  Returns false when none does.
    bool uniform_candidate(std::vector<int32_t> &best) const {
        bool found = false;
        double best_f = 0.0;
        for (int n = 1; n <= kLevels; ++n) {
            std::vector<int32_t> y(L, n);
            if (!feasible(y)) continue;
            const double f = accuracy(y);
            if (!found || f > best_f) best = y, best_f = f, found = true;
        }
        return found;
    }

    // Random move of the candidate towards the budget: passes over the
    // layers, each in a fresh random order (Fisher-Yates), densifying each
    // visited layer by one level when the result still meets the budget,
    // until a pass changes nothing.
    void randomise_towards_target(std::vector<int32_t> &y) {
        for (;;) {
            std::vector<int> order(L);
            for (int l = 0; l < L; ++l) order[l] = l;
            for (int j = 0; j + 1 < L; ++j) {
                const int r = j + rng.below(L - j);
                std::swap(order[j], order[r]);
            }
            bool changed = false;
            for (int l : order) {
                if (y[l] >= kLevels) continue;
                ++y[l];
                if (feasible(y))
                    changed = true;
                else
                    --y[l];
            }
            if (!changed) return;
        }
    }

    // One offspring of parent x by overshoot, repair and refine.
    std::vector<int32_t> offspring(const std::vector<int32_t> &x, int overshoot) {
        std::vector<int32_t> y = x;
        // overshoot: densify `overshoot` distinct random layers that are not dense
        std::vector<int> U;
        for (int l = 0; l < L; ++l)
            if (y[l] < kLevels) U.push_back(l);
        const int K = overshoot < (int)U.size() ? overshoot : (int)U.size();
        for (int j = 0; j < K; ++j) {
            const int r = j + rng.below((int)U.size() - j);
            std::swap(U[j], U[r]);
            ++y[U[j]];
        }
        // repair: sparsify random layers until the budget holds
        while (!feasible(y)) {
            std::vector<int> V;
            for (int l = 0; l < L; ++l)
                if (y[l] > 1) V.push_back(l);
            if (V.empty()) return y;  // cannot be repaired: stays infeasible
            --y[V[rng.below((int)V.size())]];
        }
        // refine: densify random layers whose densification keeps the
        // budget and does not lower the fitness, while there are any
        for (;;) {
            const double base = accuracy(y);
            std::vector<int> D;
            for (int l = 0; l < L; ++l) {
                if (y[l] >= kLevels) continue;
                ++y[l];
                if (feasible(y) && accuracy(y) >= base) D.push_back(l);
                --y[l];
            }
            if (D.empty()) return y;
            ++y[D[rng.below((int)D.size())]];
        }
    }
};

}  // namespace

extern "C" nm_status nm_search(int layers, const double *lut, const double *gamma, double b, double target,
                               nm_fitness_fn fitness, void *user, const nm_search_params *p, int32_t *best,
                               double *best_fitness, double *trace) {
    if (layers < 1 || !lut || !gamma || !fitness || !p || !best) return NM_ERR_ARG;
    if (p->generations < 0 || p->offspring < 1 || p->overshoot < 1 || p->reserved != 0) return NM_ERR_ARG;
    for (int64_t i = 0; i < (int64_t)layers * kLevels; ++i)
        if (!std::isfinite(lut[i])) return NM_ERR_ARG;
    Search s{layers, lut, gamma, b, target, fitness, user, CounterRng{p->seed}};

    std::vector<int32_t> x;
    if (!s.uniform_candidate(x)) return NM_ERR_SHAPE;
    s.randomise_towards_target(x);
    double fx = s.fitness(x);
    for (int g = 0; g < p->generations; ++g) {
        if (trace) trace[g] = fx;
        // (1 + lambda) selection: the fittest offspring (first on ties)
        // replaces the parent unless it is less fit
        std::vector<int32_t> champion;
        double fc = -std::numeric_limits<double>::infinity();
        for (int i = 0; i < p->offspring; ++i) {
            std::vector<int32_t> y = s.offspring(x, p->overshoot);
            const double fy = s.fitness(y);
            if (champion.empty() || fy > fc) champion = y, fc = fy;
        }
        if (fc >= fx) x = champion, fx = fc;
    }
    if (trace) trace[p->generations] = fx;
    for (int l = 0; l < layers; ++l) best[l] = x[l];
    if (best_fitness) *best_fitness = fx;
    return NM_OK;
}
