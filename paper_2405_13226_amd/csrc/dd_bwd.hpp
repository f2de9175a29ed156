// dd_bwd.hpp -- pieces of the attention backward shared by its translation
// units (dd_bwd.hip: prep, dK/dV for D = 64, dQ and the launcher;
// dd_dkdv.hip: dK/dV for D = 128).
#pragma once

#include "dd_device.hpp"
#include "dd_internal.h"
#include "dd_rope.hpp"

namespace dd {

// Per-call values every backward kernel takes, derived once by the launcher.
struct BwdScalars {
    const float *lse2;   // [B*H][L] log-sum-exp in log2 units (workspace)
    const float *delta;  // [B*H][L] rowsum(dO * O) (workspace)
    float scale_log2;    // softmax scale times log2(e)
    float scale;         // softmax scale 1/sqrt(D)
    RopeEpi rt;          // rotary frequencies for the dQ / dK epilogues
    int rope;            // 0 off, 1 row positions, 2 document-local positions
};

// dK and dV for D = 128 with the paired-wave kernel (dd_dkdv.hip); returns the
// runtime's launch status.
hipError_t launch_dkdv_paired(const BwdArgs &a, const BwdScalars &s);

}  // namespace dd
