// Static device scratch of curvefp_gemm_ws_static, for callers that cannot allocate (code under
// HIP graph capture, serving loops, harnesses that forbid hipMalloc).
//
// The array lives in this translation unit alone, so its code object -- and with it the
// CURVEFP_STATIC_SCRATCH_BYTES of device memory each GPU then holds until the process ends -- is
// loaded only by a process that calls that entry point.  In host code the array's name is a
// host-side stand-in, not a device address: the address each device gives it comes from
// hipGetSymbolAddress, looked up once per device with that device current and kept here; only
// that pointer is ever handed to kernels.  Every call on one GPU shares that GPU's array.
#include <atomic>
#include <mutex>

#include "../../include/curvefp.h"
#include "curvefp_internal.hpp"

namespace curvefp {

static __device__ __align__(256) char scratch[CURVEFP_STATIC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::atomic<void*> g_scratch_ptr[MAX_DEVICES];
std::mutex g_scratch_mu;

}  // namespace

hipError_t static_scratch(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255u) != 0) return hipErrorInvalidSymbol;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

}  // namespace curvefp
