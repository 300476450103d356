// Library-owned scratch for oc_layer_cached_static: callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc) still pass inputs and outputs, and the
// workspace comes from this file-scope device array instead.  Each device
// holds its own copy of the array at its own address, taken once per device
// with hipGetSymbolAddress; host code only ever uses that address (the
// array's name in host code is not a device address).
#include "../../include/oc.h"
#include "oc_internal.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace oc {

__device__ __align__(256) unsigned char scratch[OC_STATIC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void *g_scratch[MAX_DEVICES] = {};
}  // namespace

// Address of the current device's scratch (looked up on the first call on
// that device).
hipError_t static_scratch(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr || ((uintptr_t)p & 255u)) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace oc
