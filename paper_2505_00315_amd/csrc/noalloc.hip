// Allocation-free forward: mosa_forward with its scratch memory taken from a
// file-scope device array instead of a caller buffer (for callers that cannot
// allocate device memory: code under stream capture, serving loops, harnesses
// that forbid hipMalloc).  See include/mosa.h for the contract.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"
#include "mosa.h"

namespace mosa {
size_t forward_scratch_bytes(const mosa_shape* s);
int forward_impl(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y, int accumulate,
                 int32_t* I_out, float* r_out, void* saved, size_t saved_bytes, void* scratch,
                 size_t scratch_bytes, void* stream_, mosa_stage_events* ev, bool fwd_scratch_only);
}  // namespace mosa

namespace {

// The forward's scratch.  Every GPU the library runs on holds its own copy
// (at its own address) until the process ends.  In host code the array's name
// stands for a host-side shadow, not the device memory: kernels get the
// per-device address from hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[MOSA_NOALLOC_SCRATCH_MAX];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};  // device address of `scratch` per device, set at the first call there

// Device address of the current device's copy of `scratch` (looked up once
// per device, with that device current).
int scratch_ptr(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return MOSA_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return MOSA_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOSA_ERR_HIP;
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return MOSA_OK;
}

}  // namespace

extern "C" int mosa_forward_noalloc(const mosa_shape* s, const void* X, const mosa_weights* w, void* Y,
                                    int accumulate, int32_t* I_out, float* r_out, void* saved, size_t saved_bytes,
                                    void* stream) {
    // (an invalid shape gives 0 here and is rejected by forward_impl)
    if (mosa::forward_scratch_bytes(s) > MOSA_NOALLOC_SCRATCH_MAX) return MOSA_ERR_WORKSPACE;
    void* buf = nullptr;
    const int st = scratch_ptr(&buf);
    if (st) return st;
    return mosa::forward_impl(s, X, w, Y, accumulate, I_out, r_out, saved, saved_bytes, buf,
                              MOSA_NOALLOC_SCRATCH_MAX, stream, nullptr, true);
}
