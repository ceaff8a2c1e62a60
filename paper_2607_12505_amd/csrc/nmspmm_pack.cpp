// Offline packing of N:M sparse weights into the 4:2-stream layout (host only).
//
// The paper packs each N:M window's nonzeros together with their positions in
// the window so the kernel needs no separate index gathers (Sec. 4.1-4.2), and
// builds the packed form once before deployment (Sec. 6.1).  On gfx950 the
// natural packed unit is the operand of the structured-sparse matrix
// instruction: per aligned 4-group of k, two (value, 2-bit position) slots.
// Windows of 8 are cut into their two aligned 4-groups; groups that may hold
// more than two nonzeros get a second stream of slots.  The block order below
// puts each wave's operand for one (16-row fragment, 128-wide k-step, stream)
// in 1024 + 256 contiguous bytes, one 16-byte and one 4-byte load per lane.
#include <cstring>
#include <vector>

#include "nmspmm_internal.h"

namespace {

using namespace nmspmm;

bool pattern_supported(int N, int M) {
    return (M == 4 || M == 8) && N >= 1 && N <= M;
}

int streams_for(int N, int M) {
    // At most two nonzeros in every aligned 4-group: 1:4, 2:4, 1:8, 2:8.
    (void)M;
    return N <= 2 ? 1 : 2;
}

nm_status fill_desc(int n, int k, int N, int M, nm_desc *d) {
    if (!d) return NM_ERR_ARG;
    d->bad_row = -1;
    d->bad_group = -1;
    if (n < 1 || k < 1) return NM_ERR_ARG;
    if (!pattern_supported(N, M)) return NM_ERR_UNSUPPORTED;
    if (k % M != 0 || k % 16 != 0 || n % 4 != 0) return NM_ERR_SHAPE;
    const int64_t F = (n + kFragRows - 1) / kFragRows;
    const int64_t S = (k + kKStep - 1) / kKStep;
    const int st = streams_for(N, M);
    if (F * S * st * (int64_t)kVBlock > ((int64_t)1 << 40)) return NM_ERR_SHAPE;
    d->n = n;
    d->k = k;
    d->nm_n = N;
    d->nm_m = M;
    d->streams = st;
    d->layout = NM_LAYOUT_SP42;
    d->n_frags = (int)F;
    d->k_steps = (int)S;
    d->vals_bytes = F * S * st * kVBlock;
    d->meta_bytes = F * S * st * kMBlock;
    return NM_OK;
}

}  // namespace

extern "C" nm_status nm_compress_size(int n, int k, int nm_n, int nm_m, nm_desc *desc) {
    return fill_desc(n, k, nm_n, nm_m, desc);
}

extern "C" nm_status nm_compress(const int8_t *W, int n, int k, int nm_n, int nm_m,
                                 int8_t *vals, uint8_t *meta, nm_desc *desc) {
    nm_status st = fill_desc(n, k, nm_n, nm_m, desc);
    if (st != NM_OK) return st;
    if (!W || !vals || !meta) return NM_ERR_ARG;
    // Validate the whole pattern before touching the outputs.
    for (int j = 0; j < n; ++j) {
        const int8_t *row = W + (int64_t)j * k;
        for (int g = 0; g < k / nm_m; ++g) {
            int nnz = 0;
            for (int p = 0; p < nm_m; ++p) nnz += row[g * nm_m + p] != 0;
            if (nnz > nm_n) {
                desc->bad_row = j;
                desc->bad_group = g;
                return NM_ERR_PATTERN;
            }
        }
    }
    const int F = desc->n_frags, S = desc->k_steps, Q = desc->streams;
    for (int f = 0; f < F; ++f)
        for (int s = 0; s < S; ++s)
            for (int q = 0; q < Q; ++q) {
                const int64_t b = ((int64_t)f * S + s) * Q + q;
                int8_t *vb = vals + b * kVBlock;
                uint8_t *mb = meta + b * kMBlock;
                for (int L = 0; L < 64; ++L) {
                    const int row = f * kFragRows + (L % 16);
                    uint32_t word = 0;
                    for (int g = 0; g < 8; ++g) {
                        const int k0 = s * kKStep + 32 * (L / 16) + 4 * g;
                        int8_t w4[4] = {0, 0, 0, 0};
                        if (row < n && k0 < k) std::memcpy(w4, W + (int64_t)row * k + k0, 4);
                        // slots of the group: nonzeros by position, then the
                        // smallest unused positions; all positions ascending
                        int pos[4], c = 0;
                        bool used[4] = {false, false, false, false};
                        for (int p = 0; p < 4; ++p)
                            if (w4[p] != 0) { pos[c++] = p; used[p] = true; }
                        for (int p = 0; p < 4 && c < 2 * Q; ++p)
                            if (!used[p]) { pos[c++] = p; used[p] = true; }
                        for (int a = 1; a < 2 * Q; ++a)
                            for (int z = a; z > 0 && pos[z - 1] > pos[z]; --z) {
                                int t = pos[z]; pos[z] = pos[z - 1]; pos[z - 1] = t;
                            }
                        for (int t = 0; t < 2; ++t) {
                            const int p = pos[2 * q + t];
                            vb[16 * L + 2 * g + t] = w4[p];
                            word |= (uint32_t)p << (4 * g + 2 * t);
                        }
                    }
                    std::memcpy(mb + 4 * L, &word, 4);
                }
            }
    return NM_OK;
}

extern "C" nm_status nm_decompress(const nm_desc *d, const int8_t *vals, const uint8_t *meta, int8_t *W) {
    if (!d || !vals || !meta || !W) return NM_ERR_ARG;
    nm_desc chk;
    if (fill_desc(d->n, d->k, d->nm_n, d->nm_m, &chk) != NM_OK) return NM_ERR_ARG;
    if (chk.streams != d->streams || chk.n_frags != d->n_frags || chk.k_steps != d->k_steps ||
        chk.vals_bytes != d->vals_bytes || chk.meta_bytes != d->meta_bytes || d->layout != NM_LAYOUT_SP42)
        return NM_ERR_ARG;
    const int n = d->n, k = d->k, F = d->n_frags, S = d->k_steps, Q = d->streams;
    // Decode into a scratch copy first so W is untouched on error.
    std::vector<int8_t> out((size_t)n * k, 0);
    for (int f = 0; f < F; ++f)
        for (int s = 0; s < S; ++s)
            for (int L = 0; L < 64; ++L) {
                const int row = f * kFragRows + (L % 16);
                for (int g = 0; g < 8; ++g) {
                    const int k0 = s * kKStep + 32 * (L / 16) + 4 * g;
                    int seen[4] = {0, 0, 0, 0};
                    int8_t w4[4] = {0, 0, 0, 0};
                    for (int q = 0; q < Q; ++q) {
                        const int64_t b = ((int64_t)f * S + s) * Q + q;
                        uint32_t word;
                        std::memcpy(&word, meta + b * kMBlock + 4 * L, 4);
                        for (int t = 0; t < 2; ++t) {
                            const int p = (word >> (4 * g + 2 * t)) & 3;
                            const int8_t v = vals[b * kVBlock + 16 * L + 2 * g + t];
                            if (v != 0) {
                                if (seen[p]) return NM_ERR_ARG;
                                seen[p] = 1;
                                w4[p] = v;
                            }
                        }
                    }
                    const bool inside = row < n && k0 < k;
                    if (!inside) {
                        if (w4[0] | w4[1] | w4[2] | w4[3]) return NM_ERR_ARG;
                        continue;
                    }
                    std::memcpy(&out[(size_t)row * k + k0], w4, 4);
                }
            }
    for (int j = 0; j < n; ++j)
        for (int g = 0; g < k / d->nm_m; ++g) {
            int nnz = 0;
            for (int p = 0; p < d->nm_m; ++p) nnz += out[(size_t)j * k + g * d->nm_m + p] != 0;
            if (nnz > d->nm_n) return NM_ERR_ARG;
        }
    std::memcpy(W, out.data(), out.size());
    return NM_OK;
}
