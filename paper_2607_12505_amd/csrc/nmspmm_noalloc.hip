// The allocation-free variant of nm_spmm_out (nm_spmm_noalloc): the split-K
// workspace of a plan -- per-tile arrival counters and int32 partial tiles --
// lives in a fixed, library-owned device array instead of a caller buffer,
// for callers that cannot allocate device memory.
//
// `scratch` below is a device symbol: in host code its name is only a
// stand-in, so every host use goes through the device address that
// hipGetSymbolAddress returns for the current device (each device holds its
// own copy of the array, at its own address).
#include <hip/hip_runtime.h>

#include <mutex>

#include "nmspmm_internal.h"

namespace nmspmm {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];  // device address of `scratch`, per device (null until set up)

// Set-up, once per device, with that device current: look up the device
// address of the array and clear its counter block (it must start at zero;
// every call leaves it at zero again).  The clear is a kernel on the caller's
// stream, ordered before the call's own launches.
nm_status scratch_for_current_device(void *stream, void **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        (void)hipGetLastError();
        return NM_ERR_HIP;
    }
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return NM_ERR_HIP;
        }
        if (launch_zero(p, kCounterBytes, stream) != 0) return NM_ERR_HIP;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return NM_OK;
}

nm_status static_workspace(size_t need, void *stream, void **ws, size_t *ws_bytes) {
    if (need > kNoAllocScratchBytes) return NM_ERR_WORKSPACE;
    void *p = nullptr;
    nm_status st = scratch_for_current_device(stream, &p);
    if (st != NM_OK) return st;
    *ws = p;
    *ws_bytes = kNoAllocScratchBytes;
    return NM_OK;
}

}  // namespace
}  // namespace nmspmm

using namespace nmspmm;

extern "C" nm_status nm_spmm_noalloc(const int8_t *X, int m, const int8_t *vals, const uint8_t *meta,
                                     const nm_desc *desc, const nm_outputs *out, void *stream, const nm_plan *plan) {
    nm_status st = check_desc(desc);
    if (st != NM_OK) return st;
    return run_gemm(kind_of(desc), X, m, vals, meta, desc->n, desc->k, desc->k_steps, desc->n_frags, out, nullptr,
                    0, stream, plan, static_workspace);
}
