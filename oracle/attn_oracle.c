/*
 * attn_oracle.c -- fp64 CPU oracle for masked causal self-attention, forward
 * and backward.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * GPU path is checked against.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no code, header, table or
 * helper with the HIP library, and it never calls into it.
 *
 * What it computes (Dataset Decomposition, arXiv 2405.13226):
 *   - A training sequence is a subsequence of one document (Sec. 2.1), and a
 *     document-masked concat-and-chunk batch forbids attention between
 *     different documents (Sec. 1; Sec. 3.6, document masking "DM").
 *   - Next-token training on a length-l sequence sees contexts of length
 *     0, 1, ..., l-1 (Appendix F, eq. avg_context), so query i attends to keys
 *     0..i of its own document, the diagonal included.
 *   - The step holds b/2^i sequences of length 2^i (Sec. 2.2); here that is
 *     the [B, L, H, D] batch.
 *   - Attention itself is the textbook softmax(scale * Q K^T) V with
 *     scale = 1/sqrt(D); the paper only cites it (Sec. 2.2).
 *
 * Mask.  For row b and positions i (query) and j (key) of that row:
 *     allowed(i, j) = (!causal || j <= i) && doc(b*L + i) == doc(b*L + j)
 * where doc(t) is the last k in [0, n_docs) with cu_doclens[k] <= t, and
 * doc(t) = 0 for every t when cu_doclens is NULL.  Offsets run over the
 * flattened B*L token axis, and attention never leaves its row b.
 *
 * Forward, per row i with A_i = { j : allowed(i, j) }:
 *     s_ij = scale * <q_i, k_j>,  m_i = max_j s_ij,  l_i = sum_j exp(s_ij - m_i)
 *     p_ij = exp(s_ij - m_i) / l_i,  o_i = sum_j p_ij v_j,  lse_i = m_i + ln l_i
 * Backward of f = sum(dO * O), through the softmax Jacobian:
 *     dv_j = sum_i p_ij dO_i,  dp_ij = <dO_i, v_j>,  delta_i = sum_j p_ij dp_ij
 *     ds_ij = p_ij (dp_ij - delta_i)
 *     dq_i = scale * sum_j ds_ij k_j,  dk_j = scale * sum_i ds_ij q_i
 * Every row has at least one allowed key (itself), so l_i > 0.
 *
 * All arithmetic is double precision.  bf16 inputs are widened exactly.
 * Layouts: q, k, v, dO are [B, L, H, D] (D innermost); lse is [B, L, H].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* bf16 bit pattern -> double, exact (bf16 is the top half of an fp32). */
static double widen_bf16(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* doc(t): the last k with cu[k] <= t, scanned literally. */
static int doc_of(long long t, const int32_t *cu, int n_docs)
{
    int d = 0;
    if (!cu)
        return 0;
    for (int k = 0; k < n_docs; ++k)
        if ((long long)cu[k] <= t)
            d = k;
    return d;
}

static int allowed(int i, int j, int causal, const int *doc)
{
    if (causal && j > i)
        return 0;
    return doc[i] == doc[j];
}

/* A (b,h) slice gathered into plain row-major [L][D] doubles. */
typedef struct {
    int L, D;
    double *q, *k, *v, *dO; /* dO may be NULL for the forward */
    int *doc;               /* doc id of every position of the row */
} slice_t;

static void slice_free(slice_t *s)
{
    free(s->q); free(s->k); free(s->v); free(s->dO); free(s->doc);
}

static long long elem_index(int b, int i, int h, int d, int L, int H, int D)
{
    return (((long long)b * L + i) * H + h) * (long long)D + d;
}

/* Gather from bf16 bit arrays (kind 0) or double arrays (kind 1). */
static int slice_gather(slice_t *s, int kind, const void *q, const void *k,
                        const void *v, const void *dO, int b, int h, int L,
                        int H, int D, const int32_t *cu, int n_docs)
{
    size_t n = (size_t)L * D;
    const void *src[4] = {q, k, v, dO};
    double **dst[4] = {&s->q, &s->k, &s->v, &s->dO};
    memset(s, 0, sizeof *s);
    s->L = L;
    s->D = D;
    for (int t = 0; t < 4; ++t) {
        if (!src[t])
            continue;
        *dst[t] = (double *)malloc(n * sizeof(double));
        if (!*dst[t])
            return -1;
        for (int i = 0; i < L; ++i)
            for (int d = 0; d < D; ++d) {
                long long e = elem_index(b, i, h, d, L, H, D);
                (*dst[t])[(size_t)i * D + d] =
                    kind == 0 ? widen_bf16(((const uint16_t *)src[t])[e])
                              : ((const double *)src[t])[e];
            }
    }
    s->doc = (int *)malloc((size_t)L * sizeof(int));
    if (!s->doc)
        return -1;
    for (int i = 0; i < L; ++i)
        s->doc[i] = doc_of((long long)b * L + i, cu, n_docs);
    return 0;
}

static double dot(const double *a, const double *b, int D)
{
    double acc = 0.0;
    for (int d = 0; d < D; ++d)
        acc += a[d] * b[d];
    return acc;
}

/* Row statistics of row i: m_i (max score) and l_i (sum of exp(s - m)).
 * srow receives s_ij for allowed j (other entries untouched). */
static void row_stats(const slice_t *s, int i, int causal, double scale,
                      double *srow, double *m_out, double *l_out)
{
    int L = s->L, D = s->D;
    double m = -INFINITY, l = 0.0;
    for (int j = 0; j < L; ++j)
        if (allowed(i, j, causal, s->doc)) {
            srow[j] = scale * dot(s->q + (size_t)i * D, s->k + (size_t)j * D, D);
            if (srow[j] > m)
                m = srow[j];
        }
    for (int j = 0; j < L; ++j)
        if (allowed(i, j, causal, s->doc))
            l += exp(srow[j] - m);
    *m_out = m;
    *l_out = l;
}

/* Forward of one row: o_i (D doubles) and lse_i. */
static void forward_row(const slice_t *s, int i, int causal, double scale,
                        double *srow, double *o, double *lse)
{
    int L = s->L, D = s->D;
    double m, l;
    row_stats(s, i, causal, scale, srow, &m, &l);
    for (int d = 0; d < D; ++d)
        o[d] = 0.0;
    for (int j = 0; j < L; ++j)
        if (allowed(i, j, causal, s->doc)) {
            double p = exp(srow[j] - m) / l;
            for (int d = 0; d < D; ++d)
                o[d] += p * s->v[(size_t)j * D + d];
        }
    *lse = m + log(l);
}

/* Backward of one slice.  Three plain passes over the same definition:
 *   1. per row: m_i, l_i and delta_i = sum_j p_ij dp_ij
 *   2. per row: dq_i = scale * sum_j ds_ij k_j
 *   3. per key column: dk_j = scale * sum_i ds_ij q_i, dv_j = sum_i p_ij dO_i
 * Each pass re-evaluates s_ij, p_ij and dp_ij from the inputs. */
static void backward_slice(const slice_t *s, int causal, double scale,
                           double *dq, double *dk, double *dv)
{
    int L = s->L, D = s->D;
    double *m = (double *)malloc((size_t)L * sizeof(double));
    double *l = (double *)malloc((size_t)L * sizeof(double));
    double *delta = (double *)malloc((size_t)L * sizeof(double));

    #pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < L; ++i) {
        double *srow = (double *)malloc((size_t)L * sizeof(double));
        row_stats(s, i, causal, scale, srow, &m[i], &l[i]);
        double acc = 0.0;
        for (int j = 0; j < L; ++j)
            if (allowed(i, j, causal, s->doc)) {
                double p = exp(srow[j] - m[i]) / l[i];
                double dp = dot(s->dO + (size_t)i * D, s->v + (size_t)j * D, D);
                acc += p * dp;
            }
        delta[i] = acc;
        free(srow);
    }

    #pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < L; ++i) {
        double *out = dq + (size_t)i * D;
        for (int d = 0; d < D; ++d)
            out[d] = 0.0;
        for (int j = 0; j < L; ++j)
            if (allowed(i, j, causal, s->doc)) {
                double sij = scale * dot(s->q + (size_t)i * D, s->k + (size_t)j * D, D);
                double p = exp(sij - m[i]) / l[i];
                double dp = dot(s->dO + (size_t)i * D, s->v + (size_t)j * D, D);
                double ds = p * (dp - delta[i]);
                for (int d = 0; d < D; ++d)
                    out[d] += scale * ds * s->k[(size_t)j * D + d];
            }
    }

    #pragma omp parallel for schedule(dynamic, 4)
    for (int j = 0; j < L; ++j) {
        double *ok = dk + (size_t)j * D, *ov = dv + (size_t)j * D;
        for (int d = 0; d < D; ++d) {
            ok[d] = 0.0;
            ov[d] = 0.0;
        }
        for (int i = 0; i < L; ++i)
            if (allowed(i, j, causal, s->doc)) {
                double sij = scale * dot(s->q + (size_t)i * D, s->k + (size_t)j * D, D);
                double p = exp(sij - m[i]) / l[i];
                double dp = dot(s->dO + (size_t)i * D, s->v + (size_t)j * D, D);
                double ds = p * (dp - delta[i]);
                for (int d = 0; d < D; ++d) {
                    ok[d] += scale * ds * s->q[(size_t)i * D + d];
                    ov[d] += p * s->dO[(size_t)i * D + d];
                }
            }
    }
    free(m);
    free(l);
    free(delta);
}

static int check_args(int B, int L, int H, int D, const int32_t *bh, int n_bh)
{
    if (B < 1 || L < 1 || H < 1 || D < 1 || n_bh < 0)
        return -1;
    for (int p = 0; p < n_bh; ++p)
        if (bh[2 * p] < 0 || bh[2 * p] >= B || bh[2 * p + 1] < 0 || bh[2 * p + 1] >= H)
            return -1;
    return 0;
}

/* ---- forward --------------------------------------------------------------
 * kind 0: q, k, v are bf16 bit patterns; kind 1: doubles.  Both [B,L,H,D].
 * bh lists n_bh (b, h) pairs; outputs are compact per listed pair:
 *   o [n_bh][L][D], lse [n_bh][L].  Returns 0, or -1 on bad arguments. */
static int forward_any(int kind, const void *q, const void *k, const void *v,
                       int B, int L, int H, int D, int causal,
                       const int32_t *cu, int n_docs, const int32_t *bh,
                       int n_bh, double *o, double *lse)
{
    if (check_args(B, L, H, D, bh, n_bh))
        return -1;
    double scale = 1.0 / sqrt((double)D);
    int rc = 0;
    for (int p = 0; p < n_bh; ++p) {
        slice_t s;
        if (slice_gather(&s, kind, q, k, v, NULL, bh[2 * p], bh[2 * p + 1], L,
                         H, D, cu, n_docs)) {
            slice_free(&s);
            rc = -1;
            break;
        }
        double *op = o + (size_t)p * L * D, *lp = lse + (size_t)p * L;
        #pragma omp parallel for schedule(dynamic, 8)
        for (int i = 0; i < L; ++i) {
            double *srow = (double *)malloc((size_t)L * sizeof(double));
            forward_row(&s, i, causal, scale, srow, op + (size_t)i * D, lp + i);
            free(srow);
        }
        slice_free(&s);
    }
    return rc;
}

static int backward_any(int kind, const void *q, const void *k, const void *v,
                        const void *dO, int B, int L, int H, int D, int causal,
                        const int32_t *cu, int n_docs, const int32_t *bh,
                        int n_bh, double *dq, double *dk, double *dv)
{
    if (check_args(B, L, H, D, bh, n_bh))
        return -1;
    double scale = 1.0 / sqrt((double)D);
    int rc = 0;
    for (int p = 0; p < n_bh; ++p) {
        slice_t s;
        if (slice_gather(&s, kind, q, k, v, dO, bh[2 * p], bh[2 * p + 1], L, H,
                         D, cu, n_docs)) {
            slice_free(&s);
            rc = -1;
            break;
        }
        size_t off = (size_t)p * L * D;
        backward_slice(&s, causal, scale, dq + off, dk + off, dv + off);
        slice_free(&s);
    }
    return rc;
}

int oracle_attn_fwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                         int B, int L, int H, int D, int causal,
                         const int32_t *cu_doclens, int n_docs,
                         const int32_t *bh, int n_bh, double *o, double *lse)
{
    return forward_any(0, q, k, v, B, L, H, D, causal, cu_doclens, n_docs, bh,
                       n_bh, o, lse);
}

int oracle_attn_fwd_f64(const double *q, const double *k, const double *v,
                        int B, int L, int H, int D, int causal,
                        const int32_t *cu_doclens, int n_docs,
                        const int32_t *bh, int n_bh, double *o, double *lse)
{
    return forward_any(1, q, k, v, B, L, H, D, causal, cu_doclens, n_docs, bh,
                       n_bh, o, lse);
}

int oracle_attn_bwd_bf16(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                         const uint16_t *dO, int B, int L, int H, int D,
                         int causal, const int32_t *cu_doclens, int n_docs,
                         const int32_t *bh, int n_bh, double *dq, double *dk,
                         double *dv)
{
    return backward_any(0, q, k, v, dO, B, L, H, D, causal, cu_doclens, n_docs,
                        bh, n_bh, dq, dk, dv);
}

int oracle_attn_bwd_f64(const double *q, const double *k, const double *v,
                        const double *dO, int B, int L, int H, int D,
                        int causal, const int32_t *cu_doclens, int n_docs,
                        const int32_t *bh, int n_bh, double *dq, double *dk,
                        double *dv)
{
    return backward_any(1, q, k, v, dO, B, L, H, D, causal, cu_doclens, n_docs,
                        bh, n_bh, dq, dk, dv);
}

/* Number of threads the OpenMP loops above run with. */
#ifdef _OPENMP
#include <omp.h>
#endif
int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
