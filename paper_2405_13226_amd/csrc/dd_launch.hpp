// dd_launch.hpp -- typed kernel launch that reports the launch status, and the
// grid of persistent launches.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>

#include "dd_device.hpp"

namespace dd {

// Launches `kern` with exactly the kernel's parameter types (deduced from the
// kernel, so a mismatched argument fails to compile) and returns the
// runtime's status for this launch.
template <typename... P, typename... A>
inline hipError_t launch_kernel(void (*kern)(P...), dim3 grid, dim3 block, hipStream_t stream,
                                A... args)
{
    static_assert(sizeof...(P) == sizeof...(A), "argument count");
    auto typed = [&](P... p) {
        void *ptrs[] = {static_cast<void *>(&p)...};
        return hipLaunchKernel(reinterpret_cast<const void *>(kern), grid, block, ptrs, 0, stream);
    };
    return typed(static_cast<P>(args)...);
}

// Compute units of the current device, cached per device id (0 on error).
int device_cu_count();

// Workgroups of a persistent launch of kernel KERN with `block` threads: as
// many as are resident at once (the runtime's occupancy for the kernel, per
// CU, times the CU count), rounded down to a multiple of the XCD count; 0 on
// error.  The per-CU figure is cached per kernel.
template <auto KERN>
long long persistent_grid(int block)
{
    static std::atomic<int> per_cu{-1};
    int n = per_cu.load(std::memory_order_relaxed);
    if (n < 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &n, reinterpret_cast<const void *>(KERN), block, 0) != hipSuccess)
            return 0;
        per_cu.store(n, std::memory_order_relaxed);
    }
    const long long wgs = static_cast<long long>(n) * device_cu_count();
    return wgs / kXcds * kXcds;
}

}  // namespace dd
