/*
 * dd_attn.h -- C ABI of the dataset-decomposition attention hot path on
 * MI355X (gfx950).
 *
 * The operation (Dataset Decomposition, arXiv 2405.13226):
 *   A training step holds a fixed token budget.  Under dataset decomposition
 *   it is B = budget / L sequences of length L = 2^i, each a piece of a single
 *   document (Sec. 2.1 and 2.2).  Under the concat-and-chunk baseline it is
 *   fixed-length chunks of concatenated documents, and document masking stops
 *   a token from attending across a document boundary (Sec. 1; Sec. 3.6).  In
 *   both cases the hot path is causal self-attention forward and backward,
 *   where a token at context position j sees the j earlier tokens of its own
 *   document and itself (Appendix F, eq. avg_context).
 *
 * Definition computed (softmax scale = 1/sqrt(D)), for row b, query i, key j:
 *   allowed(i, j) = (!causal || j <= i) &&
 *                   (cu_doclens == NULL || doc(b*L + i) == doc(b*L + j))
 *   doc(t)        = the last k in [0, n_docs) with cu_doclens[k] <= t
 *   O[b,i,h,:]    = sum_j softmax_j(scale * <Q[b,i,h,:], K[b,j,h,:]>) V[b,j,h,:]
 *                   over allowed j
 *   LSE[b,i,h]    = natural-log log-sum-exp of the allowed scaled scores
 * The backward returns the gradients of sum(dO * O) with respect to Q, K, V.
 * Attention never crosses a batch row; a document that spans a row edge is
 * split there, as concat-and-chunk splits it.
 *
 * Layouts.  Q, K, V, O, dO, dQ, dK, dV: bf16, contiguous [B, L, H, D] with D
 * innermost (token-major).  LSE: fp32, contiguous [B, L, H].  With this layout
 * a document-masked [Bc, L] batch whose documents all have length l and the
 * DD bucket batch [Bc*L/l, l] are the same bytes.
 *
 * Supported: D in {64, 128}; any L >= 1; B, H >= 1; B*L*H < 2^31; H*D < 2^23;
 * B*H*ceil(L/128) <= 2^23 - 8 (the kernels' largest grids then stay below
 * the 2^32 work-items of one dispatch).
 * Arithmetic: bf16 inputs, fp32 accumulation (matrix cores), fp32 softmax
 * statistics; probabilities and dS are rounded to bf16 before their products.
 *
 * Ownership.  Every tensor pointer is a DEVICE pointer owned by the caller,
 * including the backward workspace.  The library allocates no device memory
 * and keeps no pointer after a call returns.  Its only state is a per-device
 * cache of the compute-unit count and a per-kernel cache of its occupancy
 * (both filled on first use, atomically) and the opt-in timing records of
 * dd_prof_enable(), so calls are thread-safe.  Work is enqueued
 * asynchronously on `stream` (a hipStream_t; NULL = the default stream);
 * outputs are valid once the caller synchronises.  A call enqueues kernel
 * launches only (no allocation, memset or synchronisation), so it can be
 * captured in a HIP graph and replayed.  dd_attn_bwd_noalloc is the one
 * exception to "no state": it uses a device array the library holds.
 *
 * Errors.  Arguments are validated on the host before anything is enqueued;
 * on error nothing is launched and outputs are untouched.  No exception
 * crosses the ABI and nothing is printed.  The contents of cu_doclens live in
 * device memory and are not read by the validator; callers check a host copy
 * with dd_doclens_check().  Malformed contents cannot make a kernel access
 * memory out of bounds, but results are then unspecified.
 */
#ifndef DD_ATTN_H
#define DD_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DD_OK = 0,
    DD_ERR_NULL = 1,      /* a required pointer is NULL                        */
    DD_ERR_SHAPE = 2,     /* B, L or H < 1, B*L*H >= 2^31, H*D >= 2^23,
                             B*H*ceil(L/128) > 2^23 - 8, or a RoPE base that
                             is not finite and > 0                            */
    DD_ERR_HEADDIM = 3,   /* D is not 64 or 128                                */
    DD_ERR_DOCLENS = 4,   /* cu_doclens / n_docs inconsistent, or bad contents */
    DD_ERR_WORKSPACE = 5, /* backward workspace missing or too small           */
    DD_ERR_ALIGN = 6,     /* a tensor pointer is not 16-byte aligned (LSE: 4)  */
    DD_ERR_ALIAS = 7,     /* an output overlaps an input or another output     */
    DD_ERR_HIP = 8,       /* the HIP runtime rejected a launch                 */
    DD_ERR_SCRATCH = 9    /* dd_attn_bwd_noalloc: shape exceeds its scratch    */
} dd_status;

/*
 * Forward.  Q, K, V: inputs [B, L, H, D] bf16.  O: output [B, L, H, D] bf16.
 * LSE: output [B, L, H] fp32, saved for the backward.
 * causal: nonzero selects the causal mask (the method's setting); zero lets a
 * query see its whole document (or row, without cu_doclens).
 * cu_doclens: NULL with n_docs == 0 for no document mask; otherwise n_docs + 1
 * int32 document start offsets over the flattened B*L token axis, with
 * cu_doclens[0] == 0, strictly increasing, cu_doclens[n_docs] == B*L.
 * stream: hipStream_t or NULL.  Returns a dd_status.
 */
int dd_attn_fwd(const void *Q, const void *K, const void *V, void *O, float *LSE,
                int B, int L, int H, int D, int causal,
                const int32_t *cu_doclens, int n_docs, void *stream);

/*
 * Backward of sum(dO * O) for the forward above (same Q, K, V, mask), given
 * its outputs O and LSE and the upstream gradient dO, all as laid out above.
 * dQ, dK, dV: outputs [B, L, H, D] bf16; every element is written.
 * workspace: device scratch of at least dd_attn_bwd_workspace_bytes(B, L, H, D)
 * bytes, 16-byte aligned, owned by the caller; its contents on entry are
 * ignored and on return are unspecified.  It must not overlap any tensor.
 * Returns a dd_status.
 */
int dd_attn_bwd(const void *Q, const void *K, const void *V, const void *O,
                const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                int B, int L, int H, int D, int causal,
                const int32_t *cu_doclens, int n_docs,
                void *workspace, size_t workspace_bytes, void *stream);

/*
 * Backward without any allocation, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight training
 * loops, harnesses that forbid allocation.  Arguments and results are those
 * of dd_attn_bwd without the workspace (same kernels, bit-identical
 * outputs).  The workspace is a 16 MiB array in device memory that the
 * library holds for the rest of the process, one copy per GPU, set up on the
 * first call on that device; nothing is allocated or freed per call.  It
 * covers every shape with B*H*L <= 2^21 (e.g. a 65,536-token step with up to
 * 32 heads); larger shapes return DD_ERR_SCRATCH before anything is
 * enqueued.  Nothing in the scratch has to start at zero, and it keeps the
 * last call's contents.  Every call on one GPU uses the same scratch: calls
 * that overlap on one device (concurrent streams, or threads without
 * ordering between them) race and give unspecified results; calls ordered
 * on one stream are safe.  Returns a dd_status.
 */
int dd_attn_bwd_noalloc(const void *Q, const void *K, const void *V, const void *O,
                        const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                        int B, int L, int H, int D, int causal,
                        const int32_t *cu_doclens, int n_docs, void *stream);

/*
 * Rotary position embedding (Sec. 3, "Positional encoding"): the paper
 * rotates queries and keys before attention with base frequency f_b (10,000,
 * or 100,000).  Y = R X for one bf16 [B, L, H, D] tensor: components (2j, 2j+1)
 * of every head vector are rotated by the angle pos * base^(-2j/D); inverse
 * != 0 applies the transposed rotation (angle negated).  pos is the token's
 * index in its row, or, with doc_positions != 0 and cu_doclens given, its
 * index from the start of its document inside the row (every document then
 * starts at position 0, like a DD sequence).  Angles are formed in double
 * precision and reduced to [-pi, pi] before an fp32 sine and cosine; Y is
 * rounded to bf16.  X == Y (in place) is allowed; otherwise X and Y must not
 * overlap.  base must be finite and > 0.  cu_doclens as for dd_attn_fwd.
 * Returns a dd_status.
 */
int dd_rope(const void *X, void *Y, int B, int L, int H, int D, float base, int inverse,
            const int32_t *cu_doclens, int n_docs, int doc_positions, void *stream);

/*
 * Forward over rotated queries and keys with the query rotation done inside
 * the attention kernel (Sec. 3, "Positional encoding"): Q holds the
 * UNROTATED queries, K the keys already rotated by dd_rope (same base,
 * cu_doclens and doc_positions).  Each query row is rotated as the kernel
 * loads it into registers, bit-identically to dd_rope, and the forward of
 * dd_attn_fwd runs over the rotated rows.  Q_rot (optional, NULL to skip):
 * output [B, L, H, D] bf16 receiving the rotated queries, which is what
 * dd_attn_bwd_rope takes; it must not overlap any other tensor.  Other
 * arguments as for dd_attn_fwd and dd_rope.  Returns a dd_status
 * (DD_ERR_SHAPE for a base that is not finite and > 0).
 */
int dd_attn_fwd_rope(const void *Q, const void *K, const void *V, void *O, float *LSE,
                     void *Q_rot, int B, int L, int H, int D, int causal,
                     const int32_t *cu_doclens, int n_docs, float rope_base, int doc_positions,
                     void *stream);

/*
 * Backward for attention over rotated queries and keys.  Q and K are the
 * rotated tensors the forward consumed (dd_rope of the raw q and k with the
 * same base, cu_doclens and doc_positions); every other argument is as for
 * dd_attn_bwd.  dQ and dK are the gradients with respect to the unrotated q
 * and k: the kernels apply the transposed rotation to their fp32 accumulators
 * before rounding to bf16.  Returns a dd_status (DD_ERR_SHAPE for a base
 * that is not finite and > 0).
 */
int dd_attn_bwd_rope(const void *Q, const void *K, const void *V, const void *O,
                     const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                     int B, int L, int H, int D, int causal,
                     const int32_t *cu_doclens, int n_docs, float rope_base,
                     int doc_positions, void *workspace, size_t workspace_bytes,
                     void *stream);

/*
 * The rest of one transformer block of the paper's OpenLM models (Sec. 3.1;
 * Appendix, Table "openlm1b": hidden dimension 2048, 16 heads, SwiGLU
 * width 5632), so that a whole block step runs in this library: its
 * projections and MLP products, its LayerNorms and the SwiGLU.  Same
 * conventions as above: device pointers owned by the caller, host-side
 * validation before anything is enqueued, asynchronous on `stream`, no
 * allocation, a dd_status return.
 *
 * dd_gemm: C[M, N] = op(A) op(B) (+ R), bf16 inputs and outputs, fp32
 * accumulation on the matrix cores, all matrices row-major with row strides
 * (elements) lda, ldb, ldc.  op(A) = A stored [M][K], or (trans_a) A^T with
 * A stored [K][M]; op(B) = B stored [K][N], or (trans_b) B^T with B stored
 * [N][K]; trans_a and trans_b are not both set.  A forward projection
 * y = x W is (x, W); its backward is dx = (dy, W^T) and dW = (x^T, dy).
 * R: NULL, or a bf16 [M][N] matrix (row stride ldc) added to the rounded
 * product before the final rounding (a residual connection); R may be C
 * itself (in-place accumulation), otherwise it must not overlap C.
 * M and N multiples of 256, K a multiple of 64 (DD_ERR_SHAPE otherwise);
 * strides multiples of 8 and pointers 16-byte aligned (DD_ERR_ALIGN).  C
 * must not overlap A or B.  workspace: fp32 scratch of
 * dd_gemm_workspace_bytes(M, N, K) bytes for the split reduction of long-K
 * products (the weight gradients); may be NULL when that is 0.
 */
int dd_gemm(const void *A, long long lda, int trans_a, const void *B, long long ldb, int trans_b,
            const void *R, void *C, long long ldc, int M, int N, int K, void *workspace,
            size_t workspace_bytes, void *stream);
size_t dd_gemm_workspace_bytes(int M, int N, int K); /* 0: none needed, or invalid */

/*
 * LayerNorm over the rows of X [rows, d] (bf16, d in {512, 1024, 2048}):
 * Y = (X - mean) / sqrt(var + eps) * w + b with the biased variance of the
 * row; w, b: bf16 [d]; mean, rstd: fp32 [rows] outputs kept for the
 * backward (rstd = 1 / sqrt(var + eps)).  eps finite and > 0.
 */
int dd_layernorm_fwd(const void *X, const void *w, const void *b, void *Y, float *mean,
                     float *rstd, int rows, int d, float eps, void *stream);
/*
 * Its backward for upstream gradient dY [rows, d]: dX [rows, d] (plus dRes,
 * an optional bf16 [rows, d] gradient added before rounding, e.g. the
 * residual branch), and the parameter gradients dw, db (bf16 [d], summed
 * over the rows).  workspace: fp32 scratch of
 * dd_layernorm_bwd_workspace_bytes(rows, d) bytes.  Outputs must not
 * overlap inputs or each other.
 */
int dd_layernorm_bwd(const void *X, const void *w, const float *mean, const float *rstd,
                     const void *dY, const void *dRes, void *dX, void *dw, void *db, int rows,
                     int d, void *workspace, size_t workspace_bytes, void *stream);
size_t dd_layernorm_bwd_workspace_bytes(int rows, int d);

/*
 * SwiGLU of the MLP, elementwise over n bf16 values (n a multiple of 8):
 * Y = silu(U) * V with silu(u) = u / (1 + exp(-u)), fp32 arithmetic; and its
 * backward dU = dY * V * silu'(U), dV = dY * silu(U).  Outputs must not
 * overlap inputs.
 */
int dd_swiglu_fwd(const void *U, const void *V, void *Y, long long n, void *stream);
int dd_swiglu_bwd(const void *U, const void *V, const void *dY, void *dU, void *dV, long long n,
                  void *stream);

/*
 * Y = X^T for a bf16 matrix X [rows, cols] (row stride ldx): Y [cols, rows]
 * (row stride ldy), Y[c][r] = X[r][c], bit-exact.  The block's forward
 * products read their weights through it (Sec. 3.1; Table "openlm1b": the
 * d x 3d, d x d, d x 5632 and 5632 x d projections), so that both operands
 * of every forward product are read row-wise.  rows, cols: multiples of 64,
 * rows * cols <= 2^36; ldx >= cols, ldy >= rows, both multiples of 8;
 * pointers 16-byte aligned; X and Y must not overlap.
 */
int dd_transpose(const void *X, long long ldx, void *Y, long long ldy, int rows, int cols,
                 void *stream);

/* Workspace bytes dd_attn_bwd needs for this shape (0 for an invalid shape). */
size_t dd_attn_bwd_workspace_bytes(int B, int L, int H, int D);

/*
 * Checks a HOST copy of cu_doclens: n_docs >= 1, cu[0] == 0, strictly
 * increasing, cu[n_docs] == total_tokens.  Returns DD_OK or DD_ERR_DOCLENS
 * (DD_ERR_NULL for a NULL pointer).
 */
int dd_doclens_check(const int32_t *host_cu_doclens, int n_docs,
                     long long total_tokens);

/* Static English text of a status code ("unknown status" otherwise). */
const char *dd_status_str(int status);

/*
 * Kernel timing (diagnostics; the method itself has no such step).
 * While enabled, every kernel the library enqueues is bracketed by a pair of
 * HIP events recorded on that kernel's own stream, so the elapsed time of
 * each launch can be read back.  The events are created and owned by the
 * library and reused across enable cycles.
 *
 * dd_prof_enable(1) discards earlier records and starts recording;
 * dd_prof_enable(0) stops recording and keeps the records.
 * dd_prof_read(kernel, &total_ms, &launches) waits for the recorded events
 * of that kernel and returns the sum of their elapsed times and the number of
 * launches; kernel ids are 0 forward, 1 the one-kernel backward of D = 64
 * rows of at most 256 tokens without RoPE, 2 backward dK/dV, 3 backward dQ
 * (which also forms delta and the log2 LSE), 4 rotary embedding.  Returns
 * DD_OK, DD_ERR_NULL for a NULL output pointer, DD_ERR_SHAPE for an unknown
 * kernel id, or DD_ERR_HIP if the runtime fails.  These calls are serialised
 * internally.
 */
int dd_prof_enable(int on);
int dd_prof_read(int kernel, double *total_ms, long long *launches);
/*
 * Every recorded launch in launch order: kernels[i] receives its kernel id
 * and ms[i] its elapsed time, for the first min(capacity, recorded)
 * launches since dd_prof_enable(1); *count receives the number recorded
 * (kernels and ms may be NULL when capacity is 0).  Waits for the events it
 * reads.  Returns DD_OK, DD_ERR_NULL or DD_ERR_HIP.
 */
int dd_prof_launches(int *kernels, double *ms, long long capacity, long long *count);
const char *dd_prof_kernel_name(int kernel); /* NULL for an unknown id */

#ifdef __cplusplus
}
#endif

#endif /* DD_ATTN_H */
