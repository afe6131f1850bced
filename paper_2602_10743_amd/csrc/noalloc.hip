// kla_backward_noalloc: kla_backward with its workspace in a file-scope device
// array instead of a caller-provided buffer, for callers that cannot allocate.
//
// The array `scratch` exists once per GPU the library runs on, for the life of
// the process.  In host code its name is not a device address: the address of a
// device's copy is taken once per device, with that device current, by
// hipGetSymbolAddress, and only that address is handed to the kernels.  Every
// call on one GPU shares that GPU's copy, so calls that overlap on one GPU (on
// different streams, or from different threads) race on it; calls on one stream
// are ordered by the stream.
#include <mutex>

#include <hip/hip_runtime.h>

#include "kla.h"

namespace {

__device__ __align__(256) unsigned char scratch[KLA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];
hipError_t g_status[kMaxDevices];
std::once_flag g_once[kMaxDevices];

// The address of the current device's copy of `scratch`, looked up on the first call
// on that device; NULL if the lookup failed.
void* device_scratch() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(g_once[dev], [dev] {
        void* ptr = nullptr;
        g_status[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch[dev] = g_status[dev] == hipSuccess ? ptr : nullptr;
    });
    return g_scratch[dev];
}

}  // namespace

extern "C" kla_status kla_backward_noalloc(const kla_desc* desc, const void* q, const void* k, const void* v,
                                           const void* abar, const void* pbar, const void* r, const float* lam0,
                                           const float* eta0, const void* saved, const void* dy, const float* dyvar,
                                           const float* dlamT, const float* detaT, void* dq, void* dk, void* dv,
                                           void* dabar, void* dpbar, void* dr, float* dlam0, float* deta0,
                                           hipStream_t stream) {
    if (!desc) return KLA_ERR_NULL;
    if (!saved && desc->T > 0) return KLA_ERR_NULL;   // the context is not recomputed here
    if (kla_backward_workspace(desc, 1) > (size_t)KLA_NOALLOC_SCRATCH_BYTES) return KLA_ERR_WORKSPACE;
    void* ws = device_scratch();
    if (!ws) return KLA_ERR_HIP;
    return kla_backward(desc, q, k, v, abar, pbar, r, lam0, eta0, saved, dy, dyvar, dlamT, detaT, dq, dk, dv, dabar,
                        dpbar, dr, dlam0, deta0, ws, (size_t)KLA_NOALLOC_SCRATCH_BYTES, stream);
}
