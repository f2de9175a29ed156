// dd_noalloc.hip -- the device-resident scratch behind dd_attn_bwd_noalloc.
//
// The backward needs a workspace for the log2-LSE and -delta rows (fp32
// [B*H][L] each).  dd_attn_bwd takes it from the caller; the no-allocation
// entry point uses this file-scope device array instead.  Every GPU the
// library runs on holds its own copy, at its own address, from the first
// call on that device until the process ends.  In host code the array's
// name is only a stand-in for the symbol: the device address comes from
// hipGetSymbolAddress, once per device, and is what the launches receive.
#include <hip/hip_runtime.h>

#include <atomic>

#include "dd_attn.h"
#include "dd_internal.h"

namespace dd {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

int noalloc_scratch(void **ptr)
{
    constexpr int kMaxDevices = 64;
    static std::atomic<void *> cache[kMaxDevices];
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return DD_ERR_HIP;
    if (dev < kMaxDevices) {
        void *p = cache[dev].load(std::memory_order_acquire);
        if (p != nullptr) {
            *ptr = p;
            return DD_OK;
        }
    }
    // The current device is `dev`: the address returned is that device's copy.
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
        return DD_ERR_HIP;
    if (dev < kMaxDevices)
        cache[dev].store(p, std::memory_order_release);
    *ptr = p;
    return DD_OK;
}

}  // namespace dd
