// dd_prof.hpp -- opt-in per-kernel timing with HIP events (dd_prof_* ABI).
#pragma once

#include <hip/hip_runtime.h>

namespace dd {

// The backward's delta / log2-LSE pass runs inside dQ (or inside the one-kernel
// backward of short rows), so it has no id of its own.
enum KernelId { K_FWD = 0, K_BWD_SHORT = 1, K_DKDV = 2, K_DQ = 3, K_ROPE = 4, K_COUNT = 5 };

// Brackets one launch: records a start event on `stream` at construction and
// a stop event at destruction, when timing is enabled (no-op otherwise).
class ProfScope {
public:
    ProfScope(KernelId id, hipStream_t stream);
    ~ProfScope();
    ProfScope(const ProfScope &) = delete;
    ProfScope &operator=(const ProfScope &) = delete;

private:
    int slot_;
    hipStream_t stream_;
};

}  // namespace dd
