// Measurement and test aids declared in nmprobe.h: the matrix-instruction
// rate loop, the single-instruction layout probe and the store-only run of a
// GEMM plan.  Built as libnmprobe.so, apart from the method's library, which
// it links for the GEMM kernels that the store-only probe launches.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../nmspmm_internal.h"
#include "../../../include/nmprobe.h"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));

// Each wave keeps 8 accumulators, 8 A operands and 4 B operands in registers
// and cycles through them, so consecutive instructions are independent and
// read different registers, as in the GEMM kernels' inner loop.
template <int KIND>
__global__ __launch_bounds__(256) void k_mfma_rate(const int32_t *__restrict__ ops, int iters, int32_t *out,
                                                   int64_t *ticks) {
    const int lane = threadIdx.x & 63;
    v4i a[8], acc[8];
    v8i b[4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = *(const v4i *)(ops + (i * 64 + lane) * 4);
        acc[i] = v4i{0, 0, 0, 0};
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = *(const v8i *)(ops + 2048 + (j * 64 + lane) * 8);
    const int64_t c0 = clock64(), r0 = wall_clock64();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if constexpr (KIND == NM_KIND_SP42) {
                // position words: pairs (0,1) and (2,3) of every 4-group, alternating
                const int pos = (i & 1) ? (int)0xEEEEEEEE : 0x44444444;
                acc[i] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(a[i], b[i & 3], acc[i], pos, 0, 0);
            } else if ((i & 1) == 0) {
                // two instructions per accumulator (the two k-halves of a
                // 128-wide k-step), as in the dense GEMM kernel
                acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i], b[(i >> 1) & 3].lo, acc[i], 0, 0, 0);
                acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[i + 1], b[(i >> 1) & 3].hi, acc[i], 0, 0, 0);
            }
        }
    }
    const int64_t c1 = clock64(), r1 = wall_clock64();
    int s = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += acc[i][0] ^ acc[i][1] ^ acc[i][2] ^ acc[i][3];
    out[blockIdx.x * 256 + threadIdx.x] = s;
    if (ticks && threadIdx.x == 0) {
        ticks[2 * blockIdx.x] = c1 - c0;
        ticks[2 * blockIdx.x + 1] = r1 - r0;
    }
}

// One instruction of KIND on one wave; operands and results lane-major.
template <int KIND>
__global__ __launch_bounds__(64) void k_mfma_layout(const int32_t *__restrict__ a, const int32_t *__restrict__ b,
                                                    const int32_t *__restrict__ pos, int32_t *d) {
    const int lane = threadIdx.x;
    const v4i av = *(const v4i *)(a + lane * 4);
    v4i acc = v4i{0, 0, 0, 0};
    if constexpr (KIND == NM_KIND_SP42) {
        const v8i bv = *(const v8i *)(b + lane * 8);
        acc = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av, bv, acc, pos[lane], 0, 0);
    } else {
        const v4i bv = *(const v4i *)(b + lane * 4);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bv, acc, 0, 0, 0);
    }
    *(v4i *)(d + lane * 4) = acc;
}

}  // namespace

extern "C" nm_status nm_probe_mfma_layout(int kind, const int32_t *a, const int32_t *b, const int32_t *pos,
                                          int32_t *d, void *stream) {
    if (!a || !b || !d) return NM_ERR_ARG;
    if (kind == NM_KIND_SP42) {
        if (!pos) return NM_ERR_ARG;
        hipLaunchKernelGGL(k_mfma_layout<NM_KIND_SP42>, dim3(1), dim3(64), 0, (hipStream_t)stream, a, b, pos, d);
    } else if (kind == NM_KIND_DENSE) {
        hipLaunchKernelGGL(k_mfma_layout<NM_KIND_DENSE>, dim3(1), dim3(64), 0, (hipStream_t)stream, a, b, pos, d);
    } else {
        return NM_ERR_ARG;
    }
    return hipGetLastError() == hipSuccess ? NM_OK : NM_ERR_HIP;
}

extern "C" nm_status nm_wall_clock_khz(int32_t *khz) {
    if (!khz) return NM_ERR_ARG;
    int dev = 0, rate = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&rate, hipDeviceAttributeWallClockRate, dev) !=
                                                 hipSuccess) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    *khz = rate;
    return NM_OK;
}

extern "C" nm_status nm_probe_mfma_rate(int kind, const int32_t *operands, int iters, int workgroups, int32_t *out,
                                        int64_t *ticks, void *stream) {
    if (!operands || !out || iters < 1 || workgroups < 1) return NM_ERR_ARG;
    if (kind == NM_KIND_SP42)
        hipLaunchKernelGGL(k_mfma_rate<NM_KIND_SP42>, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, operands,
                           iters, out, ticks);
    else if (kind == NM_KIND_DENSE)
        hipLaunchKernelGGL(k_mfma_rate<NM_KIND_DENSE>, dim3(workgroups), dim3(256), 0, (hipStream_t)stream,
                           operands, iters, out, ticks);
    else
        return NM_ERR_ARG;
    return hipGetLastError() == hipSuccess ? NM_OK : NM_ERR_HIP;
}

using namespace nmspmm;

namespace {
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
}  // namespace

extern "C" nm_status nm_probe_store_only(const nm_plan *plan, int m, int n, const nm_outputs *out, void *stream) {
    if (!plan || !out) return NM_ERR_ARG;
    if (m < 0 || n < 4 || n % 4 != 0) return NM_ERR_SHAPE;
    if (m == 0) return NM_OK;
    if ((int64_t)m * n >= ((int64_t)1 << 29)) return NM_ERR_SHAPE;
    const nm_outputs o = *out;
    if (!o.y && !o.yh && !o.yq) return NM_ERR_ARG;
    if ((o.yh && !o.scale) || (o.yq && !o.qscale)) return NM_ERR_ARG;
    if ((o.y && !aligned16(o.y)) || (o.yh && !aligned16(o.yh)) || (o.yh && !aligned16(o.scale)) ||
        (o.yq && !aligned16(o.yq)) || (o.yq && !aligned16(o.qscale)))
        return NM_ERR_ARG;
    if (plan->tile < 0 || plan->tile >= kNumTiles || kTiles[plan->tile].layout != kOutSplit || plan->split_k != 1)
        return NM_ERR_ARG;
    if (!kind_is_valid(plan->kind)) return NM_ERR_ARG;
    nm_plan p = *plan;
    p.expand = 0;
    nm_status st = complete_plan(p.kind, m, n, 128, &p);
    if (st != NM_OK) return st;
    // Zero k-steps: the kernel issues no operand loads and no matrix
    // instructions; the epilogue stores the zero accumulators.  No operand
    // pointer is read.
    GemmArgs a;
    a.X = nullptr;
    a.A = nullptr;
    a.meta = nullptr;
    a.Y = o.y;
    a.Yh = o.yh;
    a.scale = o.scale;
    a.Yq = o.yq;
    a.qscale = o.qscale;
    a.counters = nullptr;
    a.partials = nullptr;
    a.m = m;
    a.n = n;
    a.k = 128;
    a.k_steps = 0;
    a.n_frags = (n + kFragRows - 1) / kFragRows;
    a.tiles_n = (n + p.tile_n - 1) / p.tile_n;
    a.tiles_m = (m + p.tile_m - 1) / p.tile_m;
    a.split_k = 1;
    a.group_rows = 0;
    return launch_gemm(p.kind, p.tile, a, p.grid, stream) == 0 ? NM_OK : NM_ERR_HIP;
}

// Timing events without the system-scope fence a default event performs when
// it completes (a write-back and invalidation of the caches): between two
// GEMMs such a fence costs microseconds and leaves the next GEMM with cold
// caches, which the GEMMs of a real sequence of layers do not see.
extern "C" nm_status nm_probe_event_create(void **event) {
    if (!event) return NM_ERR_ARG;
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    *event = (void *)e;
    return NM_OK;
}

extern "C" nm_status nm_probe_event_destroy(void *event) {
    if (!event) return NM_ERR_ARG;
    if (hipEventDestroy((hipEvent_t)event) != hipSuccess) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    return NM_OK;
}

extern "C" nm_status nm_probe_event_record(void *event, void *stream) {
    if (!event) return NM_ERR_ARG;
    if (hipEventRecord((hipEvent_t)event, (hipStream_t)stream) != hipSuccess) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    return NM_OK;
}

extern "C" nm_status nm_probe_event_elapsed_ms(float *ms, void *start, void *stop) {
    if (!ms || !start || !stop) return NM_ERR_ARG;
    if (hipEventElapsedTime(ms, (hipEvent_t)start, (hipEvent_t)stop) != hipSuccess) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    return NM_OK;
}
