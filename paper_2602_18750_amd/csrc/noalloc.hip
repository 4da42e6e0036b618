// The fixed device scratch of hill_step_noalloc, for callers that cannot
// allocate device memory: a file-scope device array that every GPU the
// library runs on holds until the process ends.  Host code never passes the
// array's name to a kernel (in host code it is only a stand-in for the
// symbol): the device address of the current GPU's copy is looked up with
// hipGetSymbolAddress, once per device with that device current, and cached.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hill_internal.h"

namespace hill {

namespace {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch(void** ptr)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *ptr = g_ptr[dev];
    return hipSuccess;
}

}  // namespace hill
