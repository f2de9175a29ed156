// dd_api.cpp -- the C ABI entry points declared in include/dd_attn.h.
//
// Host-only C++: argument validation, workspace sizing and status strings.
// Nothing here touches the GPU; the launches live in dd_fwd.hip and
// dd_bwd.hip behind the internal interface of dd_internal.h.  Every check
// runs before any launch, so an invalid call leaves all outputs untouched.
#include "dd_attn.h"
#include "dd_internal.h"

#include <cmath>
#include <cstdint>
#include <initializer_list>

namespace {

// Bound on B * H * ceil(L / 128): (2^23 - 8) workgroups of 512 work-items
// stay below 2^32 work-items.
constexpr long long kMaxBlocks = (1LL << 23) - 8;

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void *p, size_t bytes)
{
    uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return Range{a, a + bytes};
}

bool overlaps(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

bool aligned(const void *p, uintptr_t n)
{
    return (reinterpret_cast<uintptr_t>(p) & (n - 1)) == 0;
}

int check_shape(int B, int L, int H, int D)
{
    if (B < 1 || L < 1 || H < 1)
        return DD_ERR_SHAPE;
    long long rows = static_cast<long long>(B) * L * H;
    if (rows >= (1LL << 31))
        return DD_ERR_SHAPE;
    // The kernels' LDS-DMA plans hold per-lane byte offsets of up to 256 token
    // rows (row stride H * D elements) in 32 bits.
    if (static_cast<long long>(H) * D >= (1LL << 23))
        return DD_ERR_SHAPE;
    // The largest one-block-per-workgroup grids hold ceil(L/128) * B * H
    // workgroups (rounded up to a multiple of 8) of at most 512 work-items,
    // and a dispatch holds fewer than 2^32 work-items.
    if (rows / L * ((L + 127) / 128) > kMaxBlocks)
        return DD_ERR_SHAPE;
    if (D != 64 && D != 128)
        return DD_ERR_HEADDIM;
    return DD_OK;
}

int check_doc_args(const int32_t *cu, int n_docs, int B, int L)
{
    if ((cu == nullptr) != (n_docs == 0))
        return DD_ERR_DOCLENS;
    if (cu != nullptr) {
        if (n_docs < 1 || static_cast<long long>(n_docs) > static_cast<long long>(B) * L)
            return DD_ERR_DOCLENS;
        if (!aligned(cu, 4))
            return DD_ERR_ALIGN;
    }
    return DD_OK;
}

}  // namespace

extern "C" {

size_t dd_attn_bwd_workspace_bytes(int B, int L, int H, int D)
{
    if (check_shape(B, L, H, D) != DD_OK)
        return 0;
    return dd::bwd_workspace_bytes(B, L, H);
}

int dd_doclens_check(const int32_t *cu, int n_docs, long long total_tokens)
{
    if (cu == nullptr)
        return DD_ERR_NULL;
    if (n_docs < 1 || total_tokens < 1 || cu[0] != 0)
        return DD_ERR_DOCLENS;
    for (int k = 0; k < n_docs; ++k)
        if (cu[k + 1] <= cu[k])
            return DD_ERR_DOCLENS;
    if (static_cast<long long>(cu[n_docs]) != total_tokens)
        return DD_ERR_DOCLENS;
    return DD_OK;
}

const char *dd_status_str(int status)
{
    switch (status) {
    case DD_OK: return "ok";
    case DD_ERR_NULL: return "a required pointer is NULL";
    case DD_ERR_SHAPE:
        return "invalid shape: need B, L, H >= 1, B*L*H < 2^31, H*D < 2^23, "
               "B*H*ceil(L/128) <= 2^23 - 8 and a RoPE base that is finite and > 0";
    case DD_ERR_HEADDIM: return "unsupported head dimension: D must be 64 or 128";
    case DD_ERR_DOCLENS: return "invalid cu_doclens / n_docs";
    case DD_ERR_WORKSPACE: return "backward workspace missing or too small";
    case DD_ERR_ALIGN: return "misaligned pointer: tensors need 16-byte alignment";
    case DD_ERR_ALIAS: return "an output buffer overlaps another buffer";
    case DD_ERR_HIP: return "HIP launch failed";
    case DD_ERR_SCRATCH:
        return "shape needs more than the 16 MiB device scratch of dd_attn_bwd_noalloc "
               "(B*H*L <= 2^21); call dd_attn_bwd with a workspace";
    default: return "unknown status";
    }
}

namespace {

int attn_fwd_checked(const void *Q, const void *K, const void *V, void *O, float *LSE, void *Qrot,
                     int B, int L, int H, int D, int causal, const int32_t *cu_doclens,
                     int n_docs, double rope_base, bool rope_doc, void *stream)
{
    if (!Q || !K || !V || !O || !LSE)
        return DD_ERR_NULL;
    int st = check_shape(B, L, H, D);
    if (st != DD_OK)
        return st;
    st = check_doc_args(cu_doclens, n_docs, B, L);
    if (st != DD_OK)
        return st;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) ||
        !aligned(LSE, 4) || (Qrot && !aligned(Qrot, 16)))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(B) * L * H * D * 2;
    const size_t lb = static_cast<size_t>(B) * L * H * 4;
    Range rq = range_of(Q, tb), rk = range_of(K, tb), rv = range_of(V, tb);
    Range ro = range_of(O, tb), rl = range_of(LSE, lb), rr = range_of(Qrot, Qrot ? tb : 0);
    for (Range in : {rq, rk, rv})
        if (overlaps(ro, in) || overlaps(rl, in) || overlaps(rr, in))
            return DD_ERR_ALIAS;
    if (overlaps(ro, rl) || overlaps(rr, ro) || overlaps(rr, rl))
        return DD_ERR_ALIAS;
    if (cu_doclens) {
        Range rc = range_of(cu_doclens, static_cast<size_t>(n_docs + 1) * 4);
        if (overlaps(rc, ro) || overlaps(rc, rl) || overlaps(rc, rr))
            return DD_ERR_ALIAS;
    }
    dd::FwdArgs a{Q, K, V, O, LSE, B, L, H, D, causal != 0, cu_doclens, n_docs, stream};
    a.rope_base = rope_base;
    a.rope_doc = rope_doc;
    a.Qrot = Qrot;
    return dd::launch_fwd(a);
}

bool valid_base(float base) { return std::isfinite(base) && base > 0.0f; }

}  // namespace

int dd_attn_fwd(const void *Q, const void *K, const void *V, void *O, float *LSE,
                int B, int L, int H, int D, int causal,
                const int32_t *cu_doclens, int n_docs, void *stream)
{
    return attn_fwd_checked(Q, K, V, O, LSE, nullptr, B, L, H, D, causal, cu_doclens, n_docs,
                            0.0, false, stream);
}

int dd_attn_fwd_rope(const void *Q, const void *K, const void *V, void *O, float *LSE,
                     void *Q_rot, int B, int L, int H, int D, int causal,
                     const int32_t *cu_doclens, int n_docs, float rope_base, int doc_positions,
                     void *stream)
{
    if (!valid_base(rope_base))
        return DD_ERR_SHAPE;
    return attn_fwd_checked(Q, K, V, O, LSE, Q_rot, B, L, H, D, causal, cu_doclens, n_docs,
                            static_cast<double>(rope_base), doc_positions != 0, stream);
}

namespace {

int attn_bwd_checked(const void *Q, const void *K, const void *V, const void *O, const void *dO,
                     const float *LSE, void *dQ, void *dK, void *dV, int B, int L, int H, int D,
                     int causal, const int32_t *cu_doclens, int n_docs, double rope_base,
                     bool rope_doc, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!Q || !K || !V || !O || !dO || !LSE || !dQ || !dK || !dV)
        return DD_ERR_NULL;
    int st = check_shape(B, L, H, D);
    if (st != DD_OK)
        return st;
    st = check_doc_args(cu_doclens, n_docs, B, L);
    if (st != DD_OK)
        return st;
    const size_t need = dd::bwd_workspace_bytes(B, L, H);
    if (!workspace || workspace_bytes < need)
        return DD_ERR_WORKSPACE;
    for (const void *p : {Q, K, V, O, dO, static_cast<const void *>(dQ),
                          static_cast<const void *>(dK), static_cast<const void *>(dV),
                          static_cast<const void *>(workspace)})
        if (!aligned(p, 16))
            return DD_ERR_ALIGN;
    if (!aligned(LSE, 4))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(B) * L * H * D * 2;
    const size_t lb = static_cast<size_t>(B) * L * H * 4;
    Range ins[] = {range_of(Q, tb), range_of(K, tb), range_of(V, tb), range_of(O, tb),
                   range_of(dO, tb), range_of(LSE, lb),
                   range_of(cu_doclens, cu_doclens ? static_cast<size_t>(n_docs + 1) * 4 : 0)};
    Range outs[] = {range_of(dQ, tb), range_of(dK, tb), range_of(dV, tb),
                    range_of(workspace, need)};
    for (int i = 0; i < 4; ++i) {
        for (Range in : ins)
            if (overlaps(outs[i], in))
                return DD_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(outs[i], outs[j]))
                return DD_ERR_ALIAS;
    }
    dd::BwdArgs a{Q, K, V, O, dO, LSE, dQ, dK, dV, B, L, H, D, causal != 0,
                  cu_doclens, n_docs, workspace, stream};
    a.rope_base = rope_base;
    a.rope_doc = rope_doc;
    return dd::launch_bwd(a);
}

}  // namespace

int dd_attn_bwd(const void *Q, const void *K, const void *V, const void *O,
                const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                int B, int L, int H, int D, int causal,
                const int32_t *cu_doclens, int n_docs,
                void *workspace, size_t workspace_bytes, void *stream)
{
    return attn_bwd_checked(Q, K, V, O, dO, LSE, dQ, dK, dV, B, L, H, D, causal, cu_doclens,
                            n_docs, 0.0, false, workspace, workspace_bytes, stream);
}

int dd_attn_bwd_noalloc(const void *Q, const void *K, const void *V, const void *O,
                        const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                        int B, int L, int H, int D, int causal,
                        const int32_t *cu_doclens, int n_docs, void *stream)
{
    if (!Q || !K || !V || !O || !dO || !LSE || !dQ || !dK || !dV)
        return DD_ERR_NULL;
    int st = check_shape(B, L, H, D);
    if (st != DD_OK)
        return st;
    st = check_doc_args(cu_doclens, n_docs, B, L);
    if (st != DD_OK)
        return st;
    if (dd::bwd_workspace_bytes(B, L, H) > dd::kNoAllocScratchBytes)
        return DD_ERR_SCRATCH;
    void *ws = nullptr;
    st = dd::noalloc_scratch(&ws);
    if (st != DD_OK)
        return st;
    return attn_bwd_checked(Q, K, V, O, dO, LSE, dQ, dK, dV, B, L, H, D, causal, cu_doclens,
                            n_docs, 0.0, false, ws, dd::kNoAllocScratchBytes, stream);
}

int dd_attn_bwd_rope(const void *Q, const void *K, const void *V, const void *O,
                     const void *dO, const float *LSE, void *dQ, void *dK, void *dV,
                     int B, int L, int H, int D, int causal,
                     const int32_t *cu_doclens, int n_docs, float rope_base,
                     int doc_positions, void *workspace, size_t workspace_bytes,
                     void *stream)
{
    if (!valid_base(rope_base))
        return DD_ERR_SHAPE;
    return attn_bwd_checked(Q, K, V, O, dO, LSE, dQ, dK, dV, B, L, H, D, causal, cu_doclens,
                            n_docs, static_cast<double>(rope_base), doc_positions != 0,
                            workspace, workspace_bytes, stream);
}

size_t dd_gemm_workspace_bytes(int M, int N, int K)
{
    if (M < 256 || N < 256 || K < 64 || M % 256 || N % 256 || K % 64)
        return 0;
    return dd::gemm_workspace_bytes(M, N, K, dd::gemm_splits(M, N, K));
}

int dd_gemm(const void *A, long long lda, int trans_a, const void *B, long long ldb, int trans_b,
            const void *R, void *C, long long ldc, int M, int N, int K, void *workspace,
            size_t workspace_bytes, void *stream)
{
    if (!A || !B || !C)
        return DD_ERR_NULL;
    if (M < 256 || N < 256 || K < 64 || M % 256 || N % 256 || K % 64 || (trans_a && trans_b))
        return DD_ERR_SHAPE;
    const long long a_rows = trans_a ? K : M, a_cols = trans_a ? M : K;
    const long long b_rows = trans_b ? N : K, b_cols = trans_b ? K : N;
    if (lda < a_cols || ldb < b_cols || ldc < N)
        return DD_ERR_SHAPE;
    if (lda % 8 || ldb % 8 || ldc % 8 || !aligned(A, 16) || !aligned(B, 16) || !aligned(C, 16) ||
        (R && !aligned(R, 16)))
        return DD_ERR_ALIGN;
    const int splits = dd::gemm_splits(M, N, K);
    const size_t need = dd::gemm_workspace_bytes(M, N, K, splits);
    if (need && (!workspace || workspace_bytes < need))
        return DD_ERR_WORKSPACE;
    if (need && !aligned(workspace, 16))
        return DD_ERR_ALIGN;
    Range ra = range_of(A, static_cast<size_t>((a_rows - 1) * lda + a_cols) * 2);
    Range rb = range_of(B, static_cast<size_t>((b_rows - 1) * ldb + b_cols) * 2);
    const size_t cbytes = static_cast<size_t>((static_cast<long long>(M) - 1) * ldc + N) * 2;
    Range rc = range_of(C, cbytes), rr = range_of(R, R ? cbytes : 0);
    Range rw = range_of(workspace, need);
    if (overlaps(rc, ra) || overlaps(rc, rb) || overlaps(rw, ra) || overlaps(rw, rb) ||
        overlaps(rw, rc) || overlaps(rw, rr) || (R && R != C && overlaps(rr, rc)))
        return DD_ERR_ALIAS;
    dd::GemmArgs a{A, B, C, R, lda, ldb, ldc, M, N, K, trans_a != 0, trans_b != 0, splits,
                   workspace, stream};
    return dd::launch_gemm(a);
}

namespace {

int check_ln(const void *X, int rows, int d)
{
    if (!X)
        return DD_ERR_NULL;
    if (rows < 1 || (d != 512 && d != 1024 && d != 2048) ||
        static_cast<long long>(rows) * d >= (1LL << 40))
        return DD_ERR_SHAPE;
    return DD_OK;
}

}  // namespace

size_t dd_layernorm_bwd_workspace_bytes(int rows, int d)
{
    if (check_ln(reinterpret_cast<const void *>(1), rows, d) != DD_OK)
        return 0;
    return dd::layernorm_workspace_bytes(rows, d);
}

int dd_layernorm_fwd(const void *X, const void *w, const void *b, void *Y, float *mean,
                     float *rstd, int rows, int d, float eps, void *stream)
{
    int st = check_ln(X, rows, d);
    if (st != DD_OK)
        return st;
    if (!w || !b || !Y || !mean || !rstd)
        return DD_ERR_NULL;
    if (!(std::isfinite(eps) && eps > 0.0f))
        return DD_ERR_SHAPE;
    for (const void *p : std::initializer_list<const void *>{X, w, b, Y})
        if (!aligned(p, 16))
            return DD_ERR_ALIGN;
    if (!aligned(mean, 4) || !aligned(rstd, 4))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(rows) * d * 2, vb = static_cast<size_t>(d) * 2,
                 sb = static_cast<size_t>(rows) * 4;
    Range ins[] = {range_of(X, tb), range_of(w, vb), range_of(b, vb)};
    Range outs[] = {range_of(Y, tb), range_of(mean, sb), range_of(rstd, sb)};
    for (int i = 0; i < 3; ++i) {
        for (Range in : ins)
            if (overlaps(outs[i], in))
                return DD_ERR_ALIAS;
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i], outs[j]))
                return DD_ERR_ALIAS;
    }
    dd::LayerNormArgs a{};
    a.X = X;
    a.w = w;
    a.b = b;
    a.Y = Y;
    a.mean = mean;
    a.rstd = rstd;
    a.rows = rows;
    a.d = d;
    a.eps = eps;
    a.stream = stream;
    return dd::launch_layernorm_fwd(a);
}

int dd_layernorm_bwd(const void *X, const void *w, const float *mean, const float *rstd,
                     const void *dY, const void *dRes, void *dX, void *dw, void *db, int rows,
                     int d, void *workspace, size_t workspace_bytes, void *stream)
{
    int st = check_ln(X, rows, d);
    if (st != DD_OK)
        return st;
    if (!w || !mean || !rstd || !dY || !dX || !dw || !db)
        return DD_ERR_NULL;
    const size_t need = dd::layernorm_workspace_bytes(rows, d);
    if (!workspace || workspace_bytes < need)
        return DD_ERR_WORKSPACE;
    for (const void *p : std::initializer_list<const void *>{X, w, dY, dX, dw, db, workspace})
        if (!aligned(p, 16))
            return DD_ERR_ALIGN;
    if ((dRes && !aligned(dRes, 16)) || !aligned(mean, 4) || !aligned(rstd, 4) ||
        !aligned(dw, 2) || !aligned(db, 2))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(rows) * d * 2, vb = static_cast<size_t>(d) * 2,
                 sb = static_cast<size_t>(rows) * 4;
    Range ins[] = {range_of(X, tb), range_of(w, vb), range_of(mean, sb), range_of(rstd, sb),
                   range_of(dY, tb), range_of(dRes, dRes ? tb : 0)};
    Range outs[] = {range_of(dX, tb), range_of(dw, vb), range_of(db, vb),
                    range_of(workspace, need)};
    for (int i = 0; i < 4; ++i) {
        for (Range in : ins)
            if (overlaps(outs[i], in))
                return DD_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(outs[i], outs[j]))
                return DD_ERR_ALIAS;
    }
    dd::LayerNormArgs a{};
    a.X = X;
    a.w = w;
    a.mean_in = mean;
    a.rstd_in = rstd;
    a.dY = dY;
    a.dRes = dRes;
    a.dX = dX;
    a.dw = dw;
    a.db = db;
    a.workspace = workspace;
    a.rows = rows;
    a.d = d;
    a.stream = stream;
    return dd::launch_layernorm_bwd(a);
}

int dd_swiglu_fwd(const void *U, const void *V, void *Y, long long n, void *stream)
{
    if (!U || !V || !Y)
        return DD_ERR_NULL;
    if (n < 8 || n % 8 || n >= (1LL << 40))
        return DD_ERR_SHAPE;
    if (!aligned(U, 16) || !aligned(V, 16) || !aligned(Y, 16))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(n) * 2;
    Range ry = range_of(Y, tb);
    if (overlaps(ry, range_of(U, tb)) || overlaps(ry, range_of(V, tb)))
        return DD_ERR_ALIAS;
    dd::SwigluArgs a{U, V, nullptr, Y, nullptr, nullptr, n, false, stream};
    return dd::launch_swiglu(a);
}

int dd_swiglu_bwd(const void *U, const void *V, const void *dY, void *dU, void *dV, long long n,
                  void *stream)
{
    if (!U || !V || !dY || !dU || !dV)
        return DD_ERR_NULL;
    if (n < 8 || n % 8 || n >= (1LL << 40))
        return DD_ERR_SHAPE;
    for (const void *p : std::initializer_list<const void *>{U, V, dY, dU, dV})
        if (!aligned(p, 16))
            return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(n) * 2;
    Range ins[] = {range_of(U, tb), range_of(V, tb), range_of(dY, tb)};
    Range rdu = range_of(dU, tb), rdv = range_of(dV, tb);
    for (Range in : ins)
        if (overlaps(rdu, in) || overlaps(rdv, in))
            return DD_ERR_ALIAS;
    if (overlaps(rdu, rdv))
        return DD_ERR_ALIAS;
    dd::SwigluArgs a{U, V, dY, nullptr, dU, dV, n, true, stream};
    return dd::launch_swiglu(a);
}

int dd_transpose(const void *X, long long ldx, void *Y, long long ldy, int rows, int cols,
                 void *stream)
{
    if (!X || !Y)
        return DD_ERR_NULL;
    if (rows < 64 || cols < 64 || rows % 64 || cols % 64 ||
        static_cast<long long>(rows) * cols > (1LL << 36) || ldx < cols || ldy < rows)
        return DD_ERR_SHAPE;
    if (ldx % 8 || ldy % 8 || !aligned(X, 16) || !aligned(Y, 16))
        return DD_ERR_ALIGN;
    Range rx = range_of(X, static_cast<size_t>((static_cast<long long>(rows) - 1) * ldx + cols) * 2);
    Range ry = range_of(Y, static_cast<size_t>((static_cast<long long>(cols) - 1) * ldy + rows) * 2);
    if (overlaps(rx, ry))
        return DD_ERR_ALIAS;
    dd::TransposeArgs a{X, Y, ldx, ldy, rows, cols, stream};
    return dd::launch_transpose(a);
}

int dd_rope(const void *X, void *Y, int B, int L, int H, int D, float base, int inverse,
            const int32_t *cu_doclens, int n_docs, int doc_positions, void *stream)
{
    if (!X || !Y)
        return DD_ERR_NULL;
    int st = check_shape(B, L, H, D);
    if (st != DD_OK)
        return st;
    if (!valid_base(base))
        return DD_ERR_SHAPE;
    st = check_doc_args(cu_doclens, n_docs, B, L);
    if (st != DD_OK)
        return st;
    if (!aligned(X, 16) || !aligned(Y, 16))
        return DD_ERR_ALIGN;
    const size_t tb = static_cast<size_t>(B) * L * H * D * 2;
    Range rx = range_of(X, tb), ry = range_of(Y, tb);
    if (X != Y && overlaps(rx, ry))
        return DD_ERR_ALIAS;
    if (cu_doclens && overlaps(ry, range_of(cu_doclens, static_cast<size_t>(n_docs + 1) * 4)))
        return DD_ERR_ALIAS;
    dd::RopeArgs a{X, Y, B, L, H, D, static_cast<double>(base), inverse != 0, cu_doclens,
                   n_docs, doc_positions != 0, stream};
    return dd::launch_rope(a);
}

}  // extern "C"
