// Fixed device scratch for pace_filter_step_noalloc: the filter step's
// workspace lives in a file-scope device array instead of a caller buffer,
// for callers that cannot allocate device memory.
//
// Each device that loads the library holds its own copy of the array until
// the process ends. In host code the array's name is only a host-side stand-in:
// the device address is looked up once per device with hipGetSymbolAddress,
// with that device current, and only that address is handed to kernels.
// The filter step needs no initialised workspace (no kernel relies on zeroed
// memory or on a previous call's contents), so nothing is cleared here.
#include <mutex>

#include <hip/hip_runtime.h>

#include "../../include/pace.h"
#include "kernels.hpp"

namespace pace {

namespace {

static __device__ __align__(256) unsigned char scratch[PACE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

}  // namespace

hipError_t noalloc_scratch(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr || ((uintptr_t)p & 255u) != 0) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace pace
