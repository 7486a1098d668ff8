// The fixed device scratch array behind moa_attn_fwd_noalloc: the workspace
// of key-split calls (decode partial states, split-K prefill partial states)
// for callers that cannot allocate device memory.
//
// The array is a file-scope device variable, so every GPU the library runs on
// holds its own copy from the moment the code object is loaded until the
// process ends.  In host code its name is only a stand-in for the symbol: the
// device address is looked up with hipGetSymbolAddress, once per device and
// with that device current, and only that address is ever handed to kernels.
// Every call on one GPU shares that GPU's array, so calls that overlap on one
// GPU (different streams, or host threads racing) overwrite each other's
// partial states.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.h"

namespace moa {
namespace {

__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_addr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(hipStream_t stream, void** ptr) {
    int dev = 0;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> guard(g_lock);
    if (g_addr[dev] == nullptr) {
        int cur = 0;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* addr = nullptr;
        e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        if (addr == nullptr) return hipErrorInvalidSymbol;
        g_addr[dev] = addr;
    }
    *ptr = g_addr[dev];
    return hipSuccess;
}

}  // namespace moa
