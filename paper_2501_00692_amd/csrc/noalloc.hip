// noalloc.hip -- the device scratch array of ssm_adjoint_grad_noalloc.
//
// The array lives in the library's code object: every GPU the library runs on
// holds its own copy, at its own address, until the process ends.  Host code
// never uses the array's name as an address (in host code it is a stand-in,
// not device memory); it asks the runtime for the current device's address
// once and keeps it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace ssmk {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
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

}  // namespace ssmk
