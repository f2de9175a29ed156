// dd_launch.hpp -- typed kernel launch that reports the launch status.
#pragma once

#include <hip/hip_runtime.h>

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

}  // namespace dd
