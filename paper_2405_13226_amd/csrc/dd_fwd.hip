// dd_fwd.hip -- forward of masked causal attention (dataset decomposition
// buckets and the document-masked concat-and-chunk baseline) on gfx950.
//
// One workgroup = 4 waves = BM = 128 queries of one (b, h) slice; each wave
// owns 32 queries and keeps their Q rows in registers as matrix-core B
// operands.  The workgroup walks the key tiles (BN = 64 keys) that the mask
// allows for its queries; K (row-major) and V (transposed) tiles are staged
// in LDS, double-buffered, with the next tile's global loads in flight while
// the current one is consumed.
//
// Per wave and tile the product is computed transposed: S^T = K Q^T puts one
// query per lane column, so the softmax row max/sum is an in-lane reduction
// plus one exchange with lane l^32, and P^T stays in registers as the B
// operand of O^T += V^T P^T.  The online softmax keeps a running max m and
// sum l in fp32 (log2 domain), rescaling the O accumulator when m grows.
// Key tiles entirely outside the mask are never visited; tiles entirely
// inside it skip the element mask (only boundary tiles evaluate it).
#include "dd_device.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_prof.hpp"
#include "dd_attn.h"

namespace dd {

template <int D>
struct FwdTile {
    static constexpr int BM = 128;       // queries per workgroup
    static constexpr int BN = 64;        // keys per tile
    static constexpr int KP = D + 8;     // K tile row pitch (elements)
    static constexpr int VP = BN + 4;    // V^T tile row pitch (elements)
    static constexpr int K_ELEMS = BN * KP;
    static constexpr int V_ELEMS = D * VP;
    static constexpr int STAGE = K_ELEMS + V_ELEMS;
    static constexpr int UNITS = 2 * (BN / 4) * (D / 8);  // K and V units per tile
    static constexpr int UNITS_PER_THREAD = UNITS / 256;
    static_assert(UNITS % 256 == 0, "tile units must divide the workgroup");
};

template <int D>
__global__ void __launch_bounds__(256, 2)
fwd_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
           const uint16_t *__restrict__ V, uint16_t *__restrict__ O, float *__restrict__ LSE,
           int B, int L, int H, int causal_i, const int32_t *__restrict__ cu, int n_docs,
           float scale_log2, int nqb)
{
    using T = FwdTile<D>;
    constexpr int KK = D / 16;  // k-steps of S^T
    constexpr int DB = D / 32;  // 32-row blocks of O^T
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * T::STAGE];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;

    // Heaviest query blocks first: block id -> (query block, b*H + h).
    const int BH = B * H;
    const int bid = blockIdx.x;
    const int qb = nqb - 1 - bid / BH;
    const int bh = bid % BH;
    const int b = bh / H, h = bh % H;

    const long long rs = static_cast<long long>(H) * D;  // token stride
    const long long base = (static_cast<long long>(b) * L * H + h) * D;
    const uint16_t *Qb = Q + base, *Kb = K + base, *Vb = V + base;

    // This lane's query and its allowed keys.
    const int q0w = qb * T::BM + wave * 32;
    const int my_q = q0w + l32;
    const bool q_ok = my_q < L;
    int lo_q = 1, hi_q = 0;  // empty for padding rows
    if (q_ok)
        query_keys(b, L, my_q, causal, cu, n_docs, lo_q, hi_q);
    const bool wave_on = q0w < L;
    // Wave key range and the sub-range every query of the wave allows.
    const int lo_w = wave_min(q_ok ? lo_q : 0x7fffffff);
    const int hi_w = wave_max(q_ok ? hi_q : -1);
    const int lo_all = wave_max(q_ok ? lo_q : -1);
    const int hi_all = wave_min(q_ok ? hi_q : 0x7fffffff);
    const bool wave_full_rows = (q0w + 31) < L;  // no padding rows in the wave

    // Workgroup key range: union over its queries (monotone in the query).
    const int qf = qb * T::BM, ql = min(qb * T::BM + T::BM - 1, L - 1);
    int wlo, whi, tmp;
    query_keys(b, L, qf, causal, cu, n_docs, wlo, tmp);
    query_keys(b, L, ql, causal, cu, n_docs, tmp, whi);
    const int t_begin = wlo / T::BN, t_end = whi / T::BN;

    // Q fragments (B operand: column = query, k-slots = 8 head dims).
    bf16x8 qf8[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (q_ok)
            v = *reinterpret_cast<const u32x4 *>(Qb + my_q * rs + kk * 16 + g * 8);
        qf8[kk] = as_bf16x8(v);
    }

    f32x16 acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
        acc[db] = f32x16{};
    float m_i = -INFINITY, l_i = 0.f;

    // Stage the first tile.
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
        uint16_t *vt = ks + T::K_ELEMS;
#pragma unroll
        for (int i = 0; i < T::UNITS_PER_THREAD; ++i) {
            const int u = tid + 256 * i;
            if (u < T::UNITS / 2)
                store_unit_rows<D, T::KP>(pre[i], ks, u);
            else
                store_unit_cols<D, T::VP>(pre[i], vt, u - T::UNITS / 2);
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
            const uint16_t *vt = ks + T::K_ELEMS;
            const bool full = wave_full_rows && j0 >= lo_all && j0 + T::BN - 1 <= hi_all;

            // S^T = K Q^T for two 32-key blocks.
            f32x16 s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                s[kb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KK; ++kk) {
                    const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                        ks + (kb * 32 + l32) * T::KP + kk * 16 + g * 8));
                    s[kb] = mfma32(a, qf8[kk], s[kb]);
                }
            }

            // Scale into the log2 domain, mask boundary tiles, tile max.
            float mt = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float x = s[kb][r] * scale_log2;
                    if (!full) {
                        const int key = j0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
                        if (key < lo_q || key > hi_q)
                            x = -INFINITY;
                    }
                    s[kb][r] = x;
                    mt = fmaxf(mt, x);
                }
            mt = fmaxf(mt, __shfl_xor(mt, 32));
            const float m_new = fmaxf(m_i, mt);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = fast_exp2(m_i - m_use);
            m_i = m_new;

            float psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float p = fast_exp2(s[kb][r] - m_use);
                    s[kb][r] = p;
                    psum += p;
                }
            l_i = l_i * alpha + psum;
#pragma unroll
            for (int db = 0; db < DB; ++db)
                acc[db] *= alpha;

            // O^T += V^T P^T.  B operand (kb, t2): registers 8*t2..8*t2+7 of
            // s[kb], i.e. keys kb*32 + 16*t2 + 4g + {0..3} and the same + 8.
            bf16x8 pb[2][2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2)
                    pb[kb][t2] = pack8(s[kb], 8 * t2);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2) {
                        const uint16_t *row = vt + (db * 32 + l32) * T::VP + kb * 32 + 16 * t2 + 4 * g;
                        const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(row);
                        const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(row + 8);
                        acc[db] = mfma32(join(lo, hi), pb[kb][t2], acc[db]);
                    }
        }

        if (t < t_end)
            commit(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    if (!q_ok)
        return;
    const float l_tot = l_i + __shfl_xor(l_i, 32);
    const float inv = 1.0f / l_tot;
    uint16_t *Ob = O + base + my_q * rs;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int d = db * 32 + 8 * rg + 4 * g;
            const bf16x4 v = pack4(acc[db][4 * rg] * inv, acc[db][4 * rg + 1] * inv,
                                   acc[db][4 * rg + 2] * inv, acc[db][4 * rg + 3] * inv);
            *reinterpret_cast<bf16x4 *>(Ob + d) = v;
        }
    if (g == 0)
        LSE[(static_cast<long long>(b) * L + my_q) * H + h] = (m_i + log2f(l_tot)) * kLn2;
}

template <int D>
static int launch_fwd_d(const FwdArgs &a)
{
    const int nqb = (a.L + FwdTile<D>::BM - 1) / FwdTile<D>::BM;
    const long long blocks = static_cast<long long>(nqb) * a.B * a.H;
    const float scale_log2 = kLog2e / sqrtf(static_cast<float>(D));
    ProfScope prof(K_FWD, static_cast<hipStream_t>(a.stream));
    const hipError_t e = launch_kernel(
        fwd_kernel<D>, dim3(static_cast<unsigned>(blocks)), dim3(256),
        static_cast<hipStream_t>(a.stream), a.Q, a.K, a.V, a.O, a.LSE, a.B, a.L, a.H,
        a.causal ? 1 : 0, a.cu, a.n_docs, scale_log2, nqb);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_fwd(const FwdArgs &a)
{
    return a.D == 64 ? launch_fwd_d<64>(a) : launch_fwd_d<128>(a);
}

}  // namespace dd
