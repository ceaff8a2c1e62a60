// Offline packing of N:M sparse weights (host only).
//
// The paper packs each N:M window's nonzero values together with their
// positions in the window, so the kernel needs no separate index gathers
// (Sec. 4.1-4.2), and builds the packed form once before deployment
// (Sec. 6.1).  Here the packed form in memory is compact -- N/M of the values
// plus a few position bits per window -- and the kernels expand it on the
// fly into the operand of a matrix instruction:
//
//   layout  patterns          per window (8) or group (4)      expanded to
//   SP42    2:4               2 values, 2 x 2-bit positions   (stored as the 4:2 operand)
//   C14     1:4               1 value,  2-bit position        one 4:2 stream
//   C18     1:8               1 value,  3-bit position        one 4:2 stream
//   C28     2:8               2 values, 2 x 3-bit positions   one 4:2 stream
//   MKn     3:8, 4:8, 5:8     n values, 8-bit occupancy mask  a dense tile (dense MFMA)
//   DENSE   3:4, 4:4, 6:8 ..  W as it is (a compact form would not be smaller
//           8:8               enough to pay for the expansion)
//
// Every layout is a sequence of blocks, one per (16-row fragment, 128-wide
// k-step), in which lane L of a wave finds the part of row 16 f + L % 16 and
// columns [128 s + 32 (L / 16), +32) that it needs, in VB value bytes and MB
// position bytes at offsets L * VB and L * MB (one load each).  The exact
// formulas are in include/nmspmm.h.
#include <cstring>
#include <vector>

#include "nmspmm_internal.h"

namespace {

using namespace nmspmm;

bool pattern_supported(int N, int M) {
    return (M == 4 || M == 8) && N >= 1 && N <= M;
}

int layout_for(int N, int M) {
    if (M == 4) return N == 1 ? NM_LAYOUT_C14 : N == 2 ? NM_LAYOUT_SP42 : NM_LAYOUT_DENSE;
    switch (N) {
        case 1: return NM_LAYOUT_C18;
        case 2: return NM_LAYOUT_C28;
        case 3: return NM_LAYOUT_MK3;
        case 4: return NM_LAYOUT_MK4;
        case 5: return NM_LAYOUT_MK5;
        default: return NM_LAYOUT_DENSE;
    }
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
    const int lay = layout_for(N, M);
    if (F * S * kVBlock > ((int64_t)1 << 40)) return NM_ERR_SHAPE;
    d->n = n;
    d->k = k;
    d->nm_n = N;
    d->nm_m = M;
    d->kind = lay;  // the kernel family of a layout has the layout's number
    d->layout = lay;
    d->n_frags = (int)F;
    d->k_steps = (int)S;
    if (lay == NM_LAYOUT_DENSE) {
        d->vals_bytes = (int64_t)n * k;
        d->meta_bytes = 0;
    } else {
        d->vals_bytes = F * S * 64 * layout_lane_vbytes(lay);
        d->meta_bytes = F * S * 64 * layout_lane_mbytes(lay);
    }
    return NM_OK;
}

// Canonical slots of one window of M weights with N slots (the window holds
// at most N nonzeros; val and pos have room for 8): the nonzeros by ascending
// position, then zero-valued pads at the smallest unused positions; the N
// positions are sorted ascending.
void canonical_slots(const int8_t *win, int M, int N, int8_t *val, int *pos) {
    bool used[8] = {false, false, false, false, false, false, false, false};
    int c = 0;
    for (int p = 0; p < M; ++p)
        if (win[p] != 0) { pos[c++] = p; used[p] = true; }
    for (int p = 0; p < M && c < N; ++p)
        if (!used[p]) { pos[c++] = p; used[p] = true; }
    for (int a = 1; a < N; ++a)
        for (int z = a; z > 0 && pos[z - 1] > pos[z]; --z) {
            int t = pos[z]; pos[z] = pos[z - 1]; pos[z - 1] = t;
        }
    for (int s = 0; s < N; ++s) val[s] = win[pos[s]];
}

// The 32 weights of lane L of block (f, s): row 16 f + L % 16, columns
// [128 s + 32 (L / 16), +32), zero outside W.
void lane_weights(const int8_t *W, int n, int k, int f, int s, int L, int8_t *w32) {
    const int row = f * kFragRows + (L % 16);
    const int c0 = s * kKStep + 32 * (L / 16);
    for (int i = 0; i < 32; ++i) w32[i] = (row < n && c0 + i < k) ? W[(int64_t)row * k + c0 + i] : 0;
}

// Packs one lane's 32 weights into its value and position bytes.
void pack_lane(int lay, const int8_t *w32, int8_t *v, uint8_t *mb) {
    switch (lay) {
        case NM_LAYOUT_SP42: {
            uint32_t word = 0;
            for (int g = 0; g < 8; ++g) {
                int8_t val[8];
                int pos[8];
                canonical_slots(w32 + 4 * g, 4, 2, val, pos);
                for (int t = 0; t < 2; ++t) {
                    v[2 * g + t] = val[t];
                    word |= (uint32_t)pos[t] << (4 * g + 2 * t);
                }
            }
            std::memcpy(mb, &word, 4);
            break;
        }
        case NM_LAYOUT_C14: {
            uint16_t half = 0;
            for (int g = 0; g < 8; ++g) {
                int8_t val[8];
                int pos[8];
                canonical_slots(w32 + 4 * g, 4, 1, val, pos);
                v[g] = val[0];
                half |= (uint16_t)(pos[0] << (2 * g));
            }
            std::memcpy(mb, &half, 2);
            break;
        }
        case NM_LAYOUT_C18: {
            uint16_t half = 0;
            for (int w = 0; w < 4; ++w) {
                int8_t val[8];
                int pos[8];
                canonical_slots(w32 + 8 * w, 8, 1, val, pos);
                v[w] = val[0];
                half |= (uint16_t)(pos[0] << (3 * w));
            }
            std::memcpy(mb, &half, 2);
            break;
        }
        case NM_LAYOUT_C28: {
            uint32_t word = 0;
            for (int w = 0; w < 4; ++w) {
                int8_t val[8];
                int pos[8];
                canonical_slots(w32 + 8 * w, 8, 2, val, pos);
                for (int t = 0; t < 2; ++t) {
                    v[2 * w + t] = val[t];
                    word |= (uint32_t)pos[t] << (6 * w + 3 * t);
                }
            }
            std::memcpy(mb, &word, 4);
            break;
        }
        default: {  // MKn: n values per window, occupancy mask per window
            const int nv = layout_mask_values(lay);
            uint32_t word = 0;
            for (int w = 0; w < 4; ++w) {
                int c = 0;
                for (int p = 0; p < 8; ++p)
                    if (w32[8 * w + p] != 0) {
                        v[nv * w + c++] = w32[8 * w + p];
                        word |= 1u << (8 * w + p);
                    }
                for (; c < nv; ++c) v[nv * w + c] = 0;
            }
            std::memcpy(mb, &word, 4);
            break;
        }
    }
}

// Inverse of pack_lane; false if the bytes cannot come from any weight
// (a position out of range, two nonzeros at one position, more nonzeros in a
// window than the layout holds).  Canonical form is checked by the caller.
bool unpack_lane(int lay, const int8_t *v, const uint8_t *mb, int8_t *w32) {
    std::memset(w32, 0, 32);
    auto put = [&](int idx, int8_t val) {
        if (val == 0) return true;
        if (w32[idx] != 0) return false;
        w32[idx] = val;
        return true;
    };
    switch (lay) {
        case NM_LAYOUT_SP42: {
            uint32_t word;
            std::memcpy(&word, mb, 4);
            for (int g = 0; g < 8; ++g)
                for (int t = 0; t < 2; ++t)
                    if (!put(4 * g + ((word >> (4 * g + 2 * t)) & 3), v[2 * g + t])) return false;
            return true;
        }
        case NM_LAYOUT_C14: {
            uint16_t half;
            std::memcpy(&half, mb, 2);
            for (int g = 0; g < 8; ++g)
                if (!put(4 * g + ((half >> (2 * g)) & 3), v[g])) return false;
            return true;
        }
        case NM_LAYOUT_C18: {
            uint16_t half;
            std::memcpy(&half, mb, 2);
            if (half >> 12) return false;
            for (int w = 0; w < 4; ++w)
                if (!put(8 * w + ((half >> (3 * w)) & 7), v[w])) return false;
            return true;
        }
        case NM_LAYOUT_C28: {
            uint32_t word;
            std::memcpy(&word, mb, 4);
            if (word >> 24) return false;
            for (int w = 0; w < 4; ++w)
                for (int t = 0; t < 2; ++t)
                    if (!put(8 * w + ((word >> (6 * w + 3 * t)) & 7), v[2 * w + t])) return false;
            return true;
        }
        default: {
            const int nv = layout_mask_values(lay);
            uint32_t word;
            std::memcpy(&word, mb, 4);
            for (int w = 0; w < 4; ++w) {
                int c = 0;
                for (int p = 0; p < 8; ++p)
                    if ((word >> (8 * w + p)) & 1) {
                        if (c >= nv) return false;
                        w32[8 * w + p] = v[nv * w + c++];
                    }
            }
            return true;
        }
    }
}

}  // namespace

extern "C" nm_status nm_compress_size(int n, int k, int nm_n, int nm_m, nm_desc *desc) {
    return fill_desc(n, k, nm_n, nm_m, desc);
}

extern "C" nm_status nm_compress(const int8_t *W, int n, int k, int nm_n, int nm_m,
                                 int8_t *vals, uint8_t *meta, nm_desc *desc) {
    nm_status st = fill_desc(n, k, nm_n, nm_m, desc);
    if (st != NM_OK) return st;
    if (!W || !vals || (desc->meta_bytes > 0 && !meta)) return NM_ERR_ARG;
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
    const int lay = desc->layout;
    if (lay == NM_LAYOUT_DENSE) {
        std::memcpy(vals, W, (size_t)n * k);
        return NM_OK;
    }
    const int F = desc->n_frags, S = desc->k_steps;
    const int VB = layout_lane_vbytes(lay), MB = layout_lane_mbytes(lay);
    int8_t w32[32];
    for (int f = 0; f < F; ++f)
        for (int s = 0; s < S; ++s) {
            const int64_t b = (int64_t)f * S + s;
            for (int L = 0; L < 64; ++L) {
                lane_weights(W, n, k, f, s, L, w32);
                pack_lane(lay, w32, vals + (b * 64 + L) * VB, meta + (b * 64 + L) * MB);
            }
        }
    return NM_OK;
}

extern "C" nm_status nm_decompress(const nm_desc *d, const int8_t *vals, const uint8_t *meta, int8_t *W) {
    if (!d || !vals || !W) return NM_ERR_ARG;
    nm_desc chk;
    if (fill_desc(d->n, d->k, d->nm_n, d->nm_m, &chk) != NM_OK) return NM_ERR_ARG;
    if (chk.kind != d->kind || chk.layout != d->layout || chk.n_frags != d->n_frags || chk.k_steps != d->k_steps ||
        chk.vals_bytes != d->vals_bytes || chk.meta_bytes != d->meta_bytes)
        return NM_ERR_ARG;
    if (d->meta_bytes > 0 && !meta) return NM_ERR_ARG;
    const int n = d->n, k = d->k, lay = d->layout;
    // Decode into a scratch copy first so W is untouched on error.
    std::vector<int8_t> out((size_t)n * k, 0);
    if (lay == NM_LAYOUT_DENSE) {
        std::memcpy(out.data(), vals, out.size());
    } else {
        const int F = d->n_frags, S = d->k_steps;
        const int VB = layout_lane_vbytes(lay), MB = layout_lane_mbytes(lay);
        int8_t w32[32], v2[32];
        uint8_t m2[4];
        for (int f = 0; f < F; ++f)
            for (int s = 0; s < S; ++s)
                for (int L = 0; L < 64; ++L) {
                    const int64_t o = ((int64_t)f * S + s) * 64 + L;
                    if (!unpack_lane(lay, vals + o * VB, meta + o * MB, w32)) return NM_ERR_ARG;
                    // canonical form: packing the decoded weights gives the same bytes
                    pack_lane(lay, w32, v2, m2);
                    if (std::memcmp(v2, vals + o * VB, VB) != 0 || std::memcmp(m2, meta + o * MB, MB) != 0)
                        return NM_ERR_ARG;
                    const int row = f * kFragRows + (L % 16);
                    const int c0 = s * kKStep + 32 * (L / 16);
                    for (int i = 0; i < 32; ++i) {
                        if (row < n && c0 + i < k)
                            out[(size_t)row * k + c0 + i] = w32[i];
                        else if (w32[i] != 0)
                            return NM_ERR_ARG;  // a nonzero in the padding rows or columns
                    }
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
