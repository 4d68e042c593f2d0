// Static device scratch of tl_gemm_noalloc: the split-K partials of callers
// that cannot allocate device memory (code under graph capture, serving loops
// that forbid hipMalloc).  The array lives in this file's code object, one
// copy per GPU, from the code object's load until the process ends; host code
// never passes its name to a kernel (in host code the name is a host-side
// stand-in, not a device address) -- it takes the device address that
// hipGetSymbolAddress returns, looked up once per device with that device
// current.
#include <hip/hip_runtime.h>

#include <mutex>

#include "tl_internal.h"

namespace tl {

static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_address(float** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = static_cast<float*>(p);
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace tl
