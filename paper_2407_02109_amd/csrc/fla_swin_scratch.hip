// Static device scratch for the allocation-free backward entry point.
//
// The array below is the backward's workspace (pad-token gradient partials, wide-window dq
// shares) for callers that cannot allocate device memory.  Each device that loads the library
// holds its own copy, at its own address, until the process ends.  In host code the array's
// name is only a host-side handle: the device address comes from hipGetSymbolAddress, taken
// once per device with that device current, and that address is what the kernels receive.
#include <mutex>

#include "fla_swin_internal.h"

namespace fla {

namespace {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_address[kMaxDevices];   // device address of `scratch` per device (NULL: not taken yet)

}  // namespace

hipError_t scratch_address(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (g_address[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_address[dev] = p;
    }
    *ptr = g_address[dev];
    return hipSuccess;
}

}  // namespace fla
