// dd_internal.h -- interface between the validated C ABI (dd_api.cpp) and the
// HIP launchers (dd_fwd.hip, dd_bwd.hip).  Host-only declarations: no HIP
// types, so the validation unit stays plain C++.
#pragma once

#include <cstddef>
#include <cstdint>

namespace dd {

struct FwdArgs {
    const void *Q, *K, *V;
    void *O;
    float *LSE;
    int B, L, H, D;
    bool causal;
    const int32_t *cu;
    int n_docs;
    void *stream;
    double rope_base = 0.0;  // > 0: Q is unrotated; rotate it at its load
    bool rope_doc = false;   // document-local positions
    void *Qrot = nullptr;    // optional output: the rotated Q
};

struct BwdArgs {
    const void *Q, *K, *V, *O, *dO;
    const float *LSE;
    void *dQ, *dK, *dV;
    int B, L, H, D;
    bool causal;
    const int32_t *cu;
    int n_docs;
    void *workspace;
    void *stream;
    double rope_base = 0.0;  // > 0: Q and K are rotated; rotate dQ, dK back
    bool rope_doc = false;   // document-local positions
};

struct RopeArgs {
    const void *X;
    void *Y;
    int B, L, H, D;
    double base;
    bool inverse;
    const int32_t *cu;
    int n_docs;
    bool doc;
    void *stream;
};

// Backward scratch: per (b, h) row, LSE in log2 units and delta = rowsum(dO*O),
// both fp32 [B*H][L], each region 256-byte aligned.
inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
inline size_t bwd_workspace_bytes(int B, int L, int H)
{
    return 2 * align256(static_cast<size_t>(B) * H * L * sizeof(float));
}

// Size of the device-resident scratch of dd_attn_bwd_noalloc (dd_noalloc.hip):
// the backward workspace of every shape with B * H * L <= 2^21.
constexpr size_t kNoAllocScratchBytes = static_cast<size_t>(16) << 20;

// Device address of this device's copy of that scratch (looked up once per
// device with the device current).  Returns DD_OK or DD_ERR_HIP.
int noalloc_scratch(void **ptr);

// Both return a dd_status value (DD_OK or DD_ERR_HIP).
int launch_fwd(const FwdArgs &a);
int launch_bwd(const BwdArgs &a);
int launch_rope(const RopeArgs &a);

}  // namespace dd
