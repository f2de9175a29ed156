// dd_bwd.hip -- backward of masked causal attention on gfx950, recomputing
// the probabilities from the forward's log-sum-exp.
//
// Three launches on the caller's stream:
//   1. prep:  delta_i = sum_d dO_id O_id and LSE in log2 units, both fp32 in
//             a [B*H][L] workspace (one contiguous row per (b, h)).
//   2. dkdv:  key-resident.  One workgroup = 4 waves = 128 keys; each wave
//             keeps its 32 keys' K and V rows in registers.  It walks the
//             query tiles (64 queries) its keys are visible to and forms
//               S = Q K^T, P = exp2(S*scale*log2e - lse2), dP = dO V^T,
//               dS = P * (dP - delta),
//               dV^T += dO^T P,  dK^T += Q^T dS.
//             Q and dO tiles are staged in LDS both row-major (operands of S
//             and dP) and transposed (operands of dV^T and dK^T).
//   3. dq:    query-resident.  One workgroup = 4 waves = 128 queries; each
//             wave keeps its queries' Q and dO rows in registers, walks the
//             key tiles (64 keys) its queries see and forms
//               S^T = K Q^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T,
//             with K (row-major and transposed) and V tiles in LDS.
// Splitting dQ from dK/dV keeps every output owned by exactly one workgroup:
// no atomics, deterministic results, at the cost of recomputing S and dP.
#include "dd_device.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_prof.hpp"
#include "dd_attn.h"

namespace dd {

// ---------------------------------------------------------------------------
// 1. delta and log2-LSE
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256)
prep_kernel(const uint16_t *__restrict__ O, const uint16_t *__restrict__ dO,
            const float *__restrict__ LSE, float *__restrict__ lse2, float *__restrict__ delta,
            int B, int L, int H)
{
    constexpr int CG = D / 8;  // lanes per (token, head) row
    const long long gid = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    const long long rows = static_cast<long long>(B) * L * H;
    const long long row = gid / CG;
    const int cg = static_cast<int>(gid % CG);
    float acc = 0.f;
    if (row < rows) {
        const u32x4 o = *reinterpret_cast<const u32x4 *>(O + row * D + cg * 8);
        const u32x4 d = *reinterpret_cast<const u32x4 *>(dO + row * D + cg * 8);
        const bf16x8 ob = as_bf16x8(o), db = as_bf16x8(d);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            acc += static_cast<float>(ob[i]) * static_cast<float>(db[i]);
    }
#pragma unroll
    for (int off = CG / 2; off >= 1; off >>= 1)
        acc += __shfl_xor(acc, off);
    if (row < rows && cg == 0) {
        const int h = static_cast<int>(row % H);
        const long long tok = row / H;
        const int i = static_cast<int>(tok % L);
        const int b = static_cast<int>(tok / L);
        const long long w = (static_cast<long long>(b) * H + h) * L + i;
        delta[w] = acc;
        lse2[w] = LSE[row] * kLog2e;
    }
}

// ---------------------------------------------------------------------------
// 2. dK, dV
// ---------------------------------------------------------------------------
template <int D>
struct KvTile {
    static constexpr int BN = 128;     // keys per workgroup
    static constexpr int BM = 64;      // queries per tile
    static constexpr int RP = D + 8;   // row-major pitch
    static constexpr int TP = BM + 4;  // transposed pitch
    static constexpr int R_ELEMS = BM * RP;
    static constexpr int T_ELEMS = D * TP;
    // Q rows, dO rows, Q^T, dO^T, then lse2[BM] and delta[BM] as floats.
    static constexpr int STAGE = 2 * R_ELEMS + 2 * T_ELEMS + 2 * BM * 2;
    static constexpr int UNITS = 2 * (BM / 4) * (D / 8);
    static constexpr int UNITS_PER_THREAD = UNITS / 256;
    static_assert(UNITS % 256 == 0, "tile units must divide the workgroup");
};

template <int D>
__global__ void __launch_bounds__(256, 1)
dkdv_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
            const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
            const float *__restrict__ lse2g, const float *__restrict__ deltag,
            uint16_t *__restrict__ dK, uint16_t *__restrict__ dV, int B, int L, int H,
            int causal_i, const int32_t *__restrict__ cu, int n_docs, float scale_log2,
            float scale, int nkb)
{
    using T = KvTile<D>;
    constexpr int KK = D / 16;
    constexpr int DB = D / 32;
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * T::STAGE];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;

    // Key blocks in ascending order: under the causal mask the first blocks
    // of a row see the most queries, so the heaviest work starts first.
    const int BH = B * H;
    const int kvb = blockIdx.x / BH;
    const int bh = blockIdx.x % BH;
    const int b = bh / H, h = bh % H;

    const long long rs = static_cast<long long>(H) * D;
    const long long base = (static_cast<long long>(b) * L * H + h) * D;
    const uint16_t *Qb = Q + base, *dOb = dO + base;
    const float *lse2 = lse2g + static_cast<long long>(bh) * L;
    const float *dlt = deltag + static_cast<long long>(bh) * L;

    const int k0w = kvb * T::BN + wave * 32;
    const int my_k = k0w + l32;
    const bool k_ok = my_k < L;
    int qlo_k = 1, qhi_k = 0;
    if (k_ok)
        key_queries(b, L, my_k, causal, cu, n_docs, qlo_k, qhi_k);
    const bool wave_on = k0w < L;
    const int lo_w = wave_min(k_ok ? qlo_k : 0x7fffffff);
    const int hi_w = wave_max(k_ok ? qhi_k : -1);
    const int lo_all = wave_max(k_ok ? qlo_k : -1);
    const int hi_all = wave_min(k_ok ? qhi_k : 0x7fffffff);
    const bool wave_full_keys = (k0w + 31) < L;

    const int kf0 = kvb * T::BN, kl = min(kvb * T::BN + T::BN - 1, L - 1);
    int wlo, whi, tmp;
    key_queries(b, L, kf0, causal, cu, n_docs, wlo, tmp);
    key_queries(b, L, kl, causal, cu, n_docs, tmp, whi);
    const int t_begin = wlo / T::BM, t_end = whi / T::BM;

    // K and V rows of this lane's key (B operands: column = key).
    bf16x8 kf[KK], vf[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
        if (k_ok) {
            kv = *reinterpret_cast<const u32x4 *>(K + base + my_k * rs + kk * 16 + g * 8);
            vv = *reinterpret_cast<const u32x4 *>(V + base + my_k * rs + kk * 16 + g * 8);
        }
        kf[kk] = as_bf16x8(kv);
        vf[kk] = as_bf16x8(vv);
    }

    f32x16 dk[DB], dv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        dk[db] = f32x16{};
        dv[db] = f32x16{};
    }

    Unit4x8 pre[T::UNITS_PER_THREAD];
    float pre_f = 0.f;
    auto issue_loads = [&](int t) {
        const int i0 = t * T::BM;
#pragma unroll
        for (int i = 0; i < T::UNITS_PER_THREAD; ++i) {
            const int u = tid + 256 * i;
            if (u < T::UNITS / 2)
                load_unit<D>(pre[i], Qb, rs, i0, L, u);
            else
                load_unit<D>(pre[i], dOb, rs, i0, L, u - T::UNITS / 2);
        }
        if (tid < 2 * T::BM) {
            const int q = i0 + (tid % T::BM);
            pre_f = q < L ? (tid < T::BM ? lse2[q] : dlt[q]) : 0.f;
        }
    };
    auto commit = [&](int buf) {
        uint16_t *qs = lds + buf * T::STAGE;
        uint16_t *dos = qs + T::R_ELEMS;
        uint16_t *qt = dos + T::R_ELEMS;
        uint16_t *dot = qt + T::T_ELEMS;
        float *fs = reinterpret_cast<float *>(dot + T::T_ELEMS);
#pragma unroll
        for (int i = 0; i < T::UNITS_PER_THREAD; ++i) {
            const int u = tid + 256 * i;
            if (u < T::UNITS / 2) {
                store_unit_rows<D, T::RP>(pre[i], qs, u);
                store_unit_cols<D, T::TP>(pre[i], qt, u);
            } else {
                store_unit_rows<D, T::RP>(pre[i], dos, u - T::UNITS / 2);
                store_unit_cols<D, T::TP>(pre[i], dot, u - T::UNITS / 2);
            }
        }
        if (tid < 2 * T::BM)
            fs[tid] = pre_f;
    };

    issue_loads(t_begin);
    commit(0);
    __syncthreads();

    int buf = 0;
    for (int t = t_begin; t <= t_end; ++t) {
        if (t < t_end)
            issue_loads(t + 1);

        const int i0 = t * T::BM;
        const bool active = wave_on && i0 <= hi_w && i0 + T::BM - 1 >= lo_w;
        if (active) {
            const uint16_t *qs = lds + buf * T::STAGE;
            const uint16_t *dos = qs + T::R_ELEMS;
            const uint16_t *qt = dos + T::R_ELEMS;
            const uint16_t *dot = qt + T::T_ELEMS;
            const float *lse_s = reinterpret_cast<const float *>(dot + T::T_ELEMS);
            const float *dlt_s = lse_s + T::BM;
            const bool full = wave_full_keys && i0 >= lo_all && i0 + T::BM - 1 <= hi_all;

            // S = Q K^T and dP = dO V^T for two 32-query blocks
            // (C layout: column = this lane's key, rows = queries).
            f32x16 s[2], dp[2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                s[qb] = f32x16{};
                dp[qb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) {
                    const int off = (qb * 32 + l32) * T::RP + kk * 16 + g * 8;
                    const bf16x8 aq = as_bf16x8(*reinterpret_cast<const u32x4 *>(qs + off));
                    const bf16x8 ad = as_bf16x8(*reinterpret_cast<const u32x4 *>(dos + off));
                    s[qb] = mfma32(aq, kf[kk], s[qb]);
                    dp[qb] = mfma32(ad, vf[kk], dp[qb]);
                }
            }

            // P and dS in place (s <- P, dp <- dS).
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int rg = 0; rg < 4; ++rg) {
                    const int ql = qb * 32 + 8 * rg + 4 * g;
                    const f32x4 lz = *reinterpret_cast<const f32x4 *>(lse_s + ql);
                    const f32x4 dz = *reinterpret_cast<const f32x4 *>(dlt_s + ql);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int r = 4 * rg + e;
                        float p = fast_exp2(s[qb][r] * scale_log2 - lz[e]);
                        if (!full) {
                            const int q = i0 + ql + e;
                            if (q < qlo_k || q > qhi_k)
                                p = 0.f;
                        }
                        s[qb][r] = p;
                        dp[qb][r] = p * (dp[qb][r] - dz[e]);
                    }
                }

            // dV^T += dO^T P and dK^T += Q^T dS.  B operand (qb, t2): rows
            // 8*t2..8*t2+7 of the C layout = queries qb*32+16*t2+4g+{0..3}, +8.
            bf16x8 pb[2][2], sb[2][2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2) {
                    pb[qb][t2] = pack8(s[qb], 8 * t2);
                    sb[qb][t2] = pack8(dp[qb], 8 * t2);
                }
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2) {
                        const int off = (db * 32 + l32) * T::TP + qb * 32 + 16 * t2 + 4 * g;
                        const bf16x8 ado = join(*reinterpret_cast<const bf16x4 *>(dot + off),
                                                *reinterpret_cast<const bf16x4 *>(dot + off + 8));
                        const bf16x8 aqt = join(*reinterpret_cast<const bf16x4 *>(qt + off),
                                                *reinterpret_cast<const bf16x4 *>(qt + off + 8));
                        dv[db] = mfma32(ado, pb[qb][t2], dv[db]);
                        dk[db] = mfma32(aqt, sb[qb][t2], dk[db]);
                    }
        }

        if (t < t_end)
            commit(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    if (!k_ok)
        return;
    uint16_t *dKb = dK + base + my_k * rs;
    uint16_t *dVb = dV + base + my_k * rs;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int d = db * 32 + 8 * rg + 4 * g;
            *reinterpret_cast<bf16x4 *>(dKb + d) =
                pack4(dk[db][4 * rg] * scale, dk[db][4 * rg + 1] * scale,
                      dk[db][4 * rg + 2] * scale, dk[db][4 * rg + 3] * scale);
            *reinterpret_cast<bf16x4 *>(dVb + d) =
                pack4(dv[db][4 * rg], dv[db][4 * rg + 1], dv[db][4 * rg + 2], dv[db][4 * rg + 3]);
        }
}

// ---------------------------------------------------------------------------
// 3. dQ
// ---------------------------------------------------------------------------
template <int D>
struct QTile {
    static constexpr int BM = 128;     // queries per workgroup
    static constexpr int BN = 64;      // keys per tile
    static constexpr int RP = D + 8;
    static constexpr int TP = BN + 4;
    static constexpr int R_ELEMS = BN * RP;
    static constexpr int T_ELEMS = D * TP;
    // K rows, V rows, K^T.
    static constexpr int STAGE = 2 * R_ELEMS + T_ELEMS;
    static constexpr int UNITS = 2 * (BN / 4) * (D / 8);
    static constexpr int UNITS_PER_THREAD = UNITS / 256;
    static_assert(UNITS % 256 == 0, "tile units must divide the workgroup");
};

template <int D>
__global__ void __launch_bounds__(256, 1)
dq_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
          const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
          const float *__restrict__ lse2g, const float *__restrict__ deltag,
          uint16_t *__restrict__ dQ, int B, int L, int H, int causal_i,
          const int32_t *__restrict__ cu, int n_docs, float scale_log2, float scale, int nqb)
{
    using T = QTile<D>;
    constexpr int KK = D / 16;
    constexpr int DB = D / 32;
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * T::STAGE];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;

    const int BH = B * H;
    const int qb = nqb - 1 - static_cast<int>(blockIdx.x) / BH;
    const int bh = blockIdx.x % BH;
    const int b = bh / H, h = bh % H;

    const long long rs = static_cast<long long>(H) * D;
    const long long base = (static_cast<long long>(b) * L * H + h) * D;
    const uint16_t *Kb = K + base, *Vb = V + base;

    const int q0w = qb * T::BM + wave * 32;
    const int my_q = q0w + l32;
    const bool q_ok = my_q < L;
    int lo_q = 1, hi_q = 0;
    if (q_ok)
        query_keys(b, L, my_q, causal, cu, n_docs, lo_q, hi_q);
    const bool wave_on = q0w < L;
    const int lo_w = wave_min(q_ok ? lo_q : 0x7fffffff);
    const int hi_w = wave_max(q_ok ? hi_q : -1);
    const int lo_all = wave_max(q_ok ? lo_q : -1);
    const int hi_all = wave_min(q_ok ? hi_q : 0x7fffffff);
    const bool wave_full_rows = (q0w + 31) < L;

    const int qf0 = qb * T::BM, ql = min(qb * T::BM + T::BM - 1, L - 1);
    int wlo, whi, tmp;
    query_keys(b, L, qf0, causal, cu, n_docs, wlo, tmp);
    query_keys(b, L, ql, causal, cu, n_docs, tmp, whi);
    const int t_begin = wlo / T::BN, t_end = whi / T::BN;

    bf16x8 qf[KK], dof[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        u32x4 qv = u32x4{0u, 0u, 0u, 0u}, dv = u32x4{0u, 0u, 0u, 0u};
        if (q_ok) {
            qv = *reinterpret_cast<const u32x4 *>(Q + base + my_q * rs + kk * 16 + g * 8);
            dv = *reinterpret_cast<const u32x4 *>(dO + base + my_q * rs + kk * 16 + g * 8);
        }
        qf[kk] = as_bf16x8(qv);
        dof[kk] = as_bf16x8(dv);
    }
    const long long wrow = static_cast<long long>(bh) * L;
    const float my_lse2 = q_ok ? lse2g[wrow + my_q] : 0.f;
    const float my_delta = q_ok ? deltag[wrow + my_q] : 0.f;

    f32x16 dq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
        dq[db] = f32x16{};

    Unit4x8 pre[T::UNITS_PER_THREAD];
    auto issue_loads = [&](int t) {
        const int j0 = t * T::BN;
#pragma unroll
        for (int i = 0; i < T::UNITS_PER_THREAD; ++i) {
            const int u = tid + 256 * i;
            if (u < T::UNITS / 2)
                load_unit<D>(pre[i], Kb, rs, j0, L, u);
            else
                load_unit<D>(pre[i], Vb, rs, j0, L, u - T::UNITS / 2);
        }
    };
    auto commit = [&](int buf) {
        uint16_t *ks = lds + buf * T::STAGE;
        uint16_t *vs = ks + T::R_ELEMS;
        uint16_t *kt = vs + T::R_ELEMS;
#pragma unroll
        for (int i = 0; i < T::UNITS_PER_THREAD; ++i) {
            const int u = tid + 256 * i;
            if (u < T::UNITS / 2) {
                store_unit_rows<D, T::RP>(pre[i], ks, u);
                store_unit_cols<D, T::TP>(pre[i], kt, u);
            } else {
                store_unit_rows<D, T::RP>(pre[i], vs, u - T::UNITS / 2);
            }
        }
    };

    issue_loads(t_begin);
    commit(0);
    __syncthreads();

    int buf = 0;
    for (int t = t_begin; t <= t_end; ++t) {
        if (t < t_end)
            issue_loads(t + 1);

        const int j0 = t * T::BN;
        const bool active = wave_on && j0 <= hi_w && j0 + T::BN - 1 >= lo_w;
        if (active) {
            const uint16_t *ks = lds + buf * T::STAGE;
            const uint16_t *vs = ks + T::R_ELEMS;
            const uint16_t *kt = vs + T::R_ELEMS;
            const bool full = wave_full_rows && j0 >= lo_all && j0 + T::BN - 1 <= hi_all;

            // S^T = K Q^T and dP^T = V dO^T (column = this lane's query).
            f32x16 s[2], dp[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                s[kb] = f32x16{};
                dp[kb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) {
                    const int off = (kb * 32 + l32) * T::RP + kk * 16 + g * 8;
                    const bf16x8 ak = as_bf16x8(*reinterpret_cast<const u32x4 *>(ks + off));
                    const bf16x8 av = as_bf16x8(*reinterpret_cast<const u32x4 *>(vs + off));
                    s[kb] = mfma32(ak, qf[kk], s[kb]);
                    dp[kb] = mfma32(av, dof[kk], dp[kb]);
                }
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float p = fast_exp2(s[kb][r] * scale_log2 - my_lse2);
                    if (!full) {
                        const int key = j0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
                        if (key < lo_q || key > hi_q)
                            p = 0.f;
                    }
                    dp[kb][r] = p * (dp[kb][r] - my_delta);
                }

            // dQ^T += K^T dS^T.
            bf16x8 sb[2][2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2)
                    sb[kb][t2] = pack8(dp[kb], 8 * t2);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2) {
                        const int off = (db * 32 + l32) * T::TP + kb * 32 + 16 * t2 + 4 * g;
                        const bf16x8 a = join(*reinterpret_cast<const bf16x4 *>(kt + off),
                                              *reinterpret_cast<const bf16x4 *>(kt + off + 8));
                        dq[db] = mfma32(a, sb[kb][t2], dq[db]);
                    }
        }

        if (t < t_end)
            commit(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    if (!q_ok)
        return;
    uint16_t *dQb = dQ + base + my_q * rs;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int d = db * 32 + 8 * rg + 4 * g;
            *reinterpret_cast<bf16x4 *>(dQb + d) =
                pack4(dq[db][4 * rg] * scale, dq[db][4 * rg + 1] * scale,
                      dq[db][4 * rg + 2] * scale, dq[db][4 * rg + 3] * scale);
        }
}

// ---------------------------------------------------------------------------
template <int D>
static int launch_bwd_d(const BwdArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const size_t region = align256(static_cast<size_t>(a.B) * a.H * a.L * sizeof(float));
    float *lse2 = static_cast<float *>(a.workspace);
    float *delta = reinterpret_cast<float *>(static_cast<char *>(a.workspace) + region);
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    const float scale_log2 = scale * kLog2e;

    const long long threads = static_cast<long long>(a.B) * a.L * a.H * (D / 8);
    const unsigned pblocks = static_cast<unsigned>((threads + 255) / 256);
    hipError_t e;
    {
        ProfScope prof(K_PREP, st);
        e = launch_kernel(prep_kernel<D>, dim3(pblocks), dim3(256), st, a.O, a.dO, a.LSE, lse2,
                          delta, a.B, a.L, a.H);
    }
    if (e != hipSuccess)
        return DD_ERR_HIP;

    const int nkb = (a.L + KvTile<D>::BN - 1) / KvTile<D>::BN;
    {
        ProfScope prof(K_DKDV, st);
        e = launch_kernel(dkdv_kernel<D>, dim3(static_cast<unsigned>(nkb * a.B * a.H)), dim3(256),
                          st, a.Q, a.K, a.V, a.dO, lse2, delta, a.dK, a.dV, a.B, a.L, a.H,
                          a.causal ? 1 : 0, a.cu, a.n_docs, scale_log2, scale, nkb);
    }
    if (e != hipSuccess)
        return DD_ERR_HIP;

    const int nqb = (a.L + QTile<D>::BM - 1) / QTile<D>::BM;
    {
        ProfScope prof(K_DQ, st);
        e = launch_kernel(dq_kernel<D>, dim3(static_cast<unsigned>(nqb * a.B * a.H)), dim3(256),
                          st, a.Q, a.K, a.V, a.dO, lse2, delta, a.dQ, a.B, a.L, a.H,
                          a.causal ? 1 : 0, a.cu, a.n_docs, scale_log2, scale, nqb);
    }
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_bwd(const BwdArgs &a)
{
    return a.D == 64 ? launch_bwd_d<64>(a) : launch_bwd_d<128>(a);
}

}  // namespace dd
