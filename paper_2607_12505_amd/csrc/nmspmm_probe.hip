// Matrix-instruction rate loop and single-instruction layout probe (measurement
// and test aids, declared in nmprobe.h).
#include <hip/hip_runtime.h>

#include "../../include/nmprobe.h"

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
