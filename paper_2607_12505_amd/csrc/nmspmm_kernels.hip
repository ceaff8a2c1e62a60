// GEMM kernels of libnmspmm for gfx950 (CDNA4): Y = X W^T in int8 with int32
// accumulation, optional per-channel fp16 dequantisation.
//
// Orientation: the weight is the A operand and the activations the B operand
// of the matrix instruction, so a 16 x 16 accumulator holds 16 output channels
// x 16 tokens and each lane ends up with 4 consecutive channels of one token:
// one 16-byte store per lane into the row-major output.  This orientation is
// forced by the structured-sparse instruction, whose sparse operand is A.
//
// Dataflow of one workgroup (4 waves) over its k range, one 128-wide k-step at
// a time (paper Sec. 4.2: sparse handling confined to packed loading, the
// compute stage purely matrix-instruction based):
//   - the tile_m x 128 int8 slice of X goes global -> VGPR -> LDS, double
//     buffered, 16-byte chunks XOR-swizzled by row so the B-operand reads of
//     16 tokens hit distinct banks;
//   - the packed weight fragments of the next k-step are loaded straight from
//     global memory into VGPRs (each lane one 16-byte value load and one
//     4-byte position load per fragment and stream) while the current step
//     computes: no decode, the packed form is the operand;
//   - each wave runs FN x FM accumulators; per token fragment it reads the
//     B operand from LDS once and reuses it for all FN weight fragments.
//   - split-K (Sec. 4.3): every split runs the same code on its k range,
//     stores its int32 partial tile, and the last split to arrive at a tile
//     (atomic counter) adds the partials and runs the epilogue, so merging
//     happens once, at the end.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "nmspmm_internal.h"

namespace nmspmm {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned short v4u16 __attribute__((ext_vector_type(4)));

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Renumber them so that consecutive logical tiles -- which share the
// same rows of X -- run on the same XCD.
__device__ inline int map_block(int bid, int nwg) {
    const int xcd = bid & 7, local = bid >> 3;
    const int per = nwg >> 3, rem = nwg & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

template <int FN, int S>
struct SparseRegs {
    v4i v[FN][S];
    int ix[FN][S];
};

template <int FN>
struct DenseRegs {
    v4i lo[FN], hi[FN];
};

template <int KIND, int WN, int WM, int FN, int FM>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
    constexpr int BN = WN * FN * 16;
    constexpr int BM = WM * FM * 16;
    constexpr bool kSparse = KIND != NM_KIND_DENSE;
    constexpr int S = KIND == NM_KIND_SP42X2 ? 2 : 1;
    constexpr int XCH = BM / 32;  // 16-byte chunks of X each thread stages per k-step
    static_assert(WN * WM == 4, "4 waves per workgroup");
    using ARegs = typename std::conditional<kSparse, SparseRegs<FN, S>, DenseRegs<FN>>::type;

    __shared__ __attribute__((aligned(16))) int8_t lds[2 * BM * 128];
    __shared__ int s_last;

    const int lid = map_block(blockIdx.x, gridDim.x);
    const int tn = lid % a.tiles_n;
    const int rest = lid / a.tiles_n;
    const int split = rest % a.split_k;
    const int tm = rest / a.split_k;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wn = wave % WN, wm = wave / WN;
    const int lg = lane >> 4;
    const int tok0 = tm * BM;
    const int ch0 = tn * BN;
    const int s_begin = (int)((int64_t)split * a.k_steps / a.split_k);
    const int s_end = (int)((int64_t)(split + 1) * a.k_steps / a.split_k);

    v4i acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    v4i xr[XCH];
    auto load_x = [&](int s) {
#pragma unroll
        for (int c = 0; c < XCH; ++c) {
            const int idx = tid + 256 * c;
            const int row = idx >> 3, chunk = idx & 7;
            const int tok = tok0 + row;
            const int kk = s * 128 + chunk * 16;
            if (tok < a.m && kk < a.k)
                xr[c] = *(const v4i *)(a.X + (size_t)tok * a.k + kk);
            else
                xr[c] = v4i{0, 0, 0, 0};
        }
    };
    auto store_x = [&](int buf) {
#pragma unroll
        for (int c = 0; c < XCH; ++c) {
            const int idx = tid + 256 * c;
            const int row = idx >> 3, chunk = idx & 7;
            *(v4i *)(lds + buf * BM * 128 + row * 128 + ((chunk ^ (row & 7)) << 4)) = xr[c];
        }
    };
    auto load_a = [&](int s, ARegs &R) {
        if constexpr (kSparse) {
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int f = (ch0 >> 4) + wn * FN + i;
#pragma unroll
                for (int q = 0; q < S; ++q) {
                    if (f < a.n_frags) {
                        const size_t b = ((size_t)f * a.k_steps + s) * S + q;
                        R.v[i][q] = *(const v4i *)(a.A + b * kVBlock + lane * 16);
                        R.ix[i][q] = *(const int *)(a.meta + b * kMBlock + lane * 4);
                    } else {
                        R.v[i][q] = v4i{0, 0, 0, 0};
                        R.ix[i][q] = 0;
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int row = ch0 + (wn * FN + i) * 16 + (lane & 15);
                const int kk = s * 128 + lg * 16;
                const int8_t *p = a.A + (size_t)row * a.k + kk;
                R.lo[i] = (row < a.n && kk < a.k) ? *(const v4i *)p : v4i{0, 0, 0, 0};
                R.hi[i] = (row < a.n && kk + 64 < a.k) ? *(const v4i *)(p + 64) : v4i{0, 0, 0, 0};
            }
        }
    };
    auto compute = [&](int buf, const ARegs &R) {
        const int8_t *L = lds + buf * BM * 128;
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int r = (wm * FM + j) * 16 + (lane & 15);
            const int8_t *rowp = L + r * 128;
            const v4i blo = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
            const v4i bhi = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
            if constexpr (kSparse) {
                const v8i b = {blo[0], blo[1], blo[2], blo[3], bhi[0], bhi[1], bhi[2], bhi[3]};
#pragma unroll
                for (int i = 0; i < FN; ++i)
#pragma unroll
                    for (int q = 0; q < S; ++q)
                        acc[i][j] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(R.v[i][q], b, acc[i][j], R.ix[i][q], 0, 0);
            } else {
#pragma unroll
                for (int i = 0; i < FN; ++i) {
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(R.lo[i], blo, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(R.hi[i], bhi, acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    ARegs cur, nxt;
    load_x(s_begin);
    load_a(s_begin, cur);
    store_x(0);
    for (int s = s_begin; s < s_end; ++s) {
        const int buf = (s - s_begin) & 1;
        __syncthreads();
        const bool more = s + 1 < s_end;
        if (more) {
            load_x(s + 1);
            load_a(s + 1, nxt);
        }
        compute(buf, cur);
        if (more) {
            store_x(buf ^ 1);
            cur = nxt;
        }
    }

    auto emit = [&](int tok, int ch, const v4i &v) {
        if (a.Y) *(v4i *)(a.Y + (size_t)tok * a.n + ch) = v;
        if (a.Yh) {
            const v4f sc = *(const v4f *)(a.scale + ch);
            v4u16 h;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const _Float16 x = (_Float16)((float)v[e] * sc[e]);
                h[e] = __builtin_bit_cast(unsigned short, x);
            }
            *(v4u16 *)(a.Yh + (size_t)tok * a.n + ch) = h;
        }
    };

    if (a.split_k == 1) {
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int ch = ch0 + (wn * FN + i) * 16 + 4 * lg;
                const int tok = tok0 + (wm * FM + j) * 16 + (lane & 15);
                if (tok < a.m && ch < a.n) emit(tok, ch, acc[i][j]);
            }
        return;
    }

    // Split-K: publish this split's partial tile, then the last split to
    // arrive adds all partials (integer addition: any order gives the same
    // result) and writes the outputs.
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int ch = ch0 + (wn * FN + i) * 16 + 4 * lg;
            const int tok = tok0 + (wm * FM + j) * 16 + (lane & 15);
            if (tok < a.m && ch < a.n)
                *(v4i *)(a.partials + ((size_t)split * a.m + tok) * a.n + ch) = acc[i][j];
        }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const int tile = tm * a.tiles_n + tn;
        const int old = atomicAdd(&a.counters[tile], 1);
        const int last = old == a.split_k - 1;
        if (last) atomicExch(&a.counters[tile], 0);  // leave the counter ready for the next call
        s_last = last;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) {
            const int ch = ch0 + (wn * FN + i) * 16 + 4 * lg;
            const int tok = tok0 + (wm * FM + j) * 16 + (lane & 15);
            if (tok >= a.m || ch >= a.n) continue;
            v4i sum = acc[i][j];
            for (int sp = 0; sp < a.split_k; ++sp) {
                if (sp == split) continue;
                sum += *(const v4i *)(a.partials + ((size_t)sp * a.m + tok) * a.n + ch);
            }
            emit(tok, ch, sum);
        }
}

__global__ void k_zero(int *p, size_t n4, unsigned char *tail, int tail_bytes) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) p[i] = 0;
    if (blockIdx.x == 0 && (int)threadIdx.x < tail_bytes) tail[threadIdx.x] = 0;
}

template <int KIND, int T>
int launch_one(const GemmArgs &args, int grid, void *stream) {
    constexpr TileCfg t = kTiles[T];
    hipLaunchKernelGGL((k_gemm<KIND, t.wn, t.wm, t.fn, t.fm>), dim3(grid), dim3(kThreads), 0,
                       (hipStream_t)stream, args);
    return (int)hipGetLastError();
}

template <int KIND, int T = 0>
int launch_kind(int tile, const GemmArgs &args, int grid, void *stream) {
    if constexpr (T < kNumTiles) {
        if (tile == T) return launch_one<KIND, T>(args, grid, stream);
        return launch_kind<KIND, T + 1>(tile, args, grid, stream);
    }
    return (int)hipErrorInvalidValue;
}

}  // namespace

int launch_gemm(int kind, int tile, const GemmArgs &args, int grid, void *stream) {
    switch (kind) {
        case NM_KIND_SP42: return launch_kind<NM_KIND_SP42>(tile, args, grid, stream);
        case NM_KIND_SP42X2: return launch_kind<NM_KIND_SP42X2>(tile, args, grid, stream);
        case NM_KIND_DENSE: return launch_kind<NM_KIND_DENSE>(tile, args, grid, stream);
    }
    return (int)hipErrorInvalidValue;
}

int launch_zero(void *ptr, size_t bytes, void *stream) {
    const size_t n4 = bytes / 4;
    const int tail = (int)(bytes % 4);
    size_t blocks = (n4 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, (int *)ptr, n4,
                       (unsigned char *)ptr + n4 * 4, tail);
    return (int)hipGetLastError();
}

}  // namespace nmspmm
