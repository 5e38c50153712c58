// Forward entry point that allocates nothing (kmip_fwd_noalloc): the score +
// select pre-passes, tiled keys and work counters live in a fixed device
// array of this library instead of a caller-supplied workspace.
//
// Host code never passes `scratch` itself to a kernel: in host code the
// array's name is only a host-side stand-in for the device symbol.  The
// device address is looked up once per device with hipGetSymbolAddress (each
// GPU holds its own copy of the array) and cached here.
#include <cstdio>
#include <mutex>

#include "kmip.h"
#include "kmip_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[KMIP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first
// call on that device.
hipError_t scratch_ptr(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

kmip_status_t kmip_fwd_noalloc(const void* Q, const void* K, const void* V, int64_t N, int32_t H,
                               int32_t d, int32_t k, float scale, float* out, int32_t* topk_idx,
                               float* lse, void* stream) {
    // kmip_fwd checks every argument before the workspace and launches
    // nothing without one: called with none, it returns KMIP_ERR_WORKSPACE
    // exactly when the other arguments are valid and there is work to do.
    kmip_status_t s = kmip_fwd(Q, K, V, nullptr, 1, N, H, d, k, scale, out, topk_idx, lse, nullptr, 0,
                               stream);
    if (s != KMIP_ERR_WORKSPACE) return s;
    const size_t need = kmip_fwd_workspace_size(N, H, d, k, 1);
    if (need > (size_t)KMIP_NOALLOC_SCRATCH_BYTES)
        return kmip::record_error(KMIP_ERR_UNSUPPORTED,
                                  "kmip_fwd_noalloc: N=%lld H=%d d=%d k=%d need %zu bytes of scratch, "
                                  "more than the %zu the library holds per device; call kmip_fwd "
                                  "with a workspace",
                                  (long long)N, H, d, k, need, (size_t)KMIP_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    const hipError_t e = scratch_ptr(&ws);
    if (e != hipSuccess)
        return kmip::record_error(KMIP_ERR_HIP, "kmip_fwd_noalloc: scratch lookup: %s", hipGetErrorString(e));
    return kmip_fwd(Q, K, V, nullptr, 1, N, H, d, k, scale, out, topk_idx, lse, ws,
                    (size_t)KMIP_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
