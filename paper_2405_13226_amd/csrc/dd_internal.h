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

// C[M, N] = op(A) op(B) (dd_gemm.hip); M and N multiples of 256, K of 64.
struct GemmArgs {
    const void *A, *B;
    void *C;
    const void *R;            // optional residual added to C (bf16, row stride ldc)
    long long lda, ldb, ldc;  // row strides in elements
    int M, N, K;
    bool trans_a, trans_b;    // A stored [K][M]; B stored [N][K] (not both)
    int splits;               // K splits (1: none); > 1 needs the workspace
    void *workspace;          // fp32 [splits][M][N]
    void *stream;
};
int gemm_splits(int M, int N, int K);
size_t gemm_workspace_bytes(int M, int N, int K, int splits);
int launch_gemm(const GemmArgs &a);

// LayerNorm over rows of d elements (dd_block.hip), d in {512, 1024, 2048}.
struct LayerNormArgs {
    const void *X, *w, *b;    // [rows, d] input; weight and bias [d]
    void *Y;                  // forward output [rows, d]
    float *mean, *rstd;       // forward outputs [rows]
    const float *mean_in, *rstd_in;
    const void *dY, *dRes;    // backward input; optional residual gradient
    void *dX, *dw, *db;       // backward outputs
    void *workspace;          // fp32 column partials
    int rows, d;
    float eps;
    void *stream;
};
size_t layernorm_workspace_bytes(int rows, int d);
int launch_layernorm_fwd(const LayerNormArgs &a);
int launch_layernorm_bwd(const LayerNormArgs &a);

// SwiGLU y = silu(u) v over n elements (n a multiple of 8), and its backward.
struct SwigluArgs {
    const void *U, *V, *dY;
    void *Y, *dU, *dV;
    long long n;
    bool backward;
    void *stream;
};
int launch_swiglu(const SwigluArgs &a);

// Y [cols, rows] = X [rows, cols] transposed (bf16, rows and cols multiples
// of 64, row strides in elements).
struct TransposeArgs {
    const void *X;
    void *Y;
    long long ldx, ldy;
    int rows, cols;
    void *stream;
};
int launch_transpose(const TransposeArgs &a);

// Both return a dd_status value (DD_OK or DD_ERR_HIP).
int launch_fwd(const FwdArgs &a);
int launch_bwd(const BwdArgs &a);
int launch_rope(const RopeArgs &a);

}  // namespace dd
