// dd_dkdv.hip -- key-resident dK, dV of the attention backward for D = 128.
//
// This kernel is its own translation unit so that it can be built with its
// own machine-instruction scheduling strategy: scheduling for instruction-
// level parallelism measures ~6% faster on it at long sequences, while the
// same strategy slows the other backward and forward kernels.
#include "dd_bwd.hpp"
#include "dd_launch.hpp"
#include "dd_tile.hpp"

namespace dd {

template <int D>
struct KvTile {
    static constexpr int BN = 128;            // keys per workgroup
    static constexpr int BM = 64;             // queries per tile
    static constexpr int NW = 8;              // waves: 4 key groups x 2 roles
    static constexpr int TILE = BM * D;       // elements of a Q or dO tile
    // Q tile, dO tile, then lse2[BM] and delta[BM] as floats.
    static constexpr int STAGE = 2 * TILE + 2 * BM * 2;
    // P hand-off between the two waves of a key group: per group, 32 fp32
    // per lane (two 32-query blocks x 16 C-layout registers), 8 KiB.
    static constexpr int PBUF_FLOATS = 4 * 64 * 32;
};

// Key-resident dK/dV.  The 32 keys of a group are shared by two waves on the
// same SIMD (wave w and w + 4):
//   role A (waves 0-3): K in registers; S = Q K^T, P = exp2(S*c - lse2)
//                       (masked), P handed to role B through LDS,
//                       dV^T += dO^T P;
//   role B (waves 4-7): V in registers; dP = dO V^T, then dS = P (dP - delta),
//                       dK^T += Q^T dS.
// Each wave holds one accumulator set, so two waves fit per SIMD and one
// wave's softmax arithmetic overlaps the other's matrix products.
template <int D>
__global__ void __launch_bounds__(512, 1)
dkdv_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
            const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
            const float *__restrict__ lse2g, const float *__restrict__ deltag,
            uint16_t *__restrict__ dK, uint16_t *__restrict__ dV, int B, int L, int H,
            int causal_i, const int32_t *__restrict__ cu, int n_docs, float scale_log2,
            float scale, int nkb, RopeEpi rt, int rope)
{
    using T = KvTile<D>;
    constexpr int KK = D / 16;
    constexpr int DB = D / 32;
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * T::STAGE];
    __shared__ __attribute__((aligned(16))) float pbuf[T::PBUF_FLOATS];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const int grp = wave & 3;
    const bool role_a = wave < 4;

    // Slices grouped per XCD; key blocks in ascending order: under the
    // causal mask the first blocks of a row see the most queries, so the
    // heaviest work starts first.
    const int BH = B * H;
    int bh, kvb;
    block_slice(blockIdx.x, nkb, BH, bh, kvb);
    const int b = bh / H, h = bh % H;

    const long long rs = static_cast<long long>(H) * D;
    const long long base = (static_cast<long long>(b) * L * H + h) * D;
    const uint16_t *Qb = Q + base, *dOb = dO + base;
    const float *lse2 = lse2g + static_cast<long long>(bh) * L;
    const float *dlt = deltag + static_cast<long long>(bh) * L;

    const int k0w = kvb * T::BN + grp * 32;
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

    // Role A keeps K rows, role B keeps V rows of this lane's key
    // (B operands: column = key).
    bf16x8 kv[KK];
    {
        const uint16_t *src = (role_a ? K : V) + base + my_k * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            u32x4 v = u32x4{0u, 0u, 0u, 0u};
            if (k_ok)
                v = *reinterpret_cast<const u32x4 *>(src + kk * 16);
            kv[kk] = as_bf16x8(v);
        }
    }

    // Per-lane LDS offsets: row reads (row l32 of a 32-query block, chunk
    // 2*kk + g) and transposed reads (rows 8*hh + 4*g + e of a 16-query step,
    // columns db*32 + 16*(G&1) + 4*c), shared by the Q and dO tiles.
    int roff[KK], toff[DB][2];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        roff[kk] = tile_off<D>(l32, kk * 16 + g * 8);
    {
        const int G = lane >> 4, e = (lane & 15) >> 2, c = lane & 3;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                toff[db][hh] = tile_off<D>(8 * hh + 4 * g + e, db * 32 + 16 * (G & 1) + 4 * c);
    }
    // This lane's slot of the P hand-off buffer: [grp][reg/4][lane][4].
    float *pslot = pbuf + grp * 64 * 32 + lane * 4;

    f32x16 acc[DB];  // dV^T (role A) or dK^T (role B)
#pragma unroll
    for (int db = 0; db < DB; ++db)
        acc[db] = f32x16{};

    DmaPlan<D, T::BM, T::NW> plan;
    plan.init(rs, wave, lane);
    auto issue = [&](int t, uint16_t *stage) {
        const int i0 = t * T::BM;
        plan.issue(stage, Qb, rs, i0, L, wave, lane);
        plan.issue(stage + T::TILE, dOb, rs, i0, L, wave, lane);
        float *fs = reinterpret_cast<float *>(stage + 2 * T::TILE);
        if (wave == 0)
            dma_row_f32(fs, lse2, i0, L, lane);
        else if (wave == 1)
            dma_row_f32(fs + T::BM, dlt, i0, L, lane);
    };

    // Transposed A operand (rows of the 16-query step of (qb, t2)) times a
    // bf16 B operand, accumulated into acc.
    auto tr_products = [&](const uint16_t *tile, const bf16x8 (&bop)[2][2]) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const uint16_t *tr = tile + (qb * 32 + 16 * t2) * D;
                    const bf16x8 a = join(lds_tr4(tr + toff[db][0]), lds_tr4(tr + toff[db][1]));
                    acc[db] = mfma32(a, bop[qb][t2], acc[db]);
                }
    };

    // Row-wise products X K^T (role A, X = Q) or X V^T (role B, X = dO).
    auto row_products = [&](const uint16_t *tile, f32x16 (&c)[2]) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            c[qb] = f32x16{};
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                c[qb] = mfma32(lds_row8(tile + qb * 32 * D + roff[kk]), kv[kk], c[qb]);
        }
    };

    // Phase 1 of a tile.  Role A: S, P (masked when MASKED), P to LDS and
    // to bf16.  Role B: dP.  Phase 2 (after a barrier): role A dV, role B
    // dS and dK.
    auto body = [&](int i0, auto bufc, auto maskc, bool active) {
        constexpr int BUF = decltype(bufc)::value;
        constexpr bool MASKED = decltype(maskc)::value != 0;
        const uint16_t *qs = lds + BUF * T::STAGE;
        const uint16_t *dos = qs + T::TILE;
        const float *lse_s = reinterpret_cast<const float *>(qs + 2 * T::TILE);
        const float *dlt_s = lse_s + T::BM;
        f32x16 c[2];
        bf16x8 bop[2][2];
        if (role_a) {
            if (active) {
                row_products(qs, c);
                const int qlo_r = qlo_k - i0 - 4 * g, qhi_r = qhi_k - i0 - 4 * g;
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg) {
                        const f32x4 lz = *reinterpret_cast<const f32x4 *>(
                            lse_s + qb * 32 + 8 * rg + 4 * g);
                        f32x4 pv;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            float p = fast_exp2(fmaf(c[qb][4 * rg + e], scale_log2, -lz[e]));
                            if constexpr (MASKED) {
                                const int qr = qb * 32 + 8 * rg + e;
                                const bool ok = (qr >= qlo_r) & (qr <= qhi_r);
                                p = ok ? p : 0.f;
                            }
                            c[qb][4 * rg + e] = p;
                            pv[e] = p;
                        }
                        *reinterpret_cast<f32x4 *>(pslot + (qb * 4 + rg) * 256) = pv;
                    }
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2)
                        bop[qb][t2] = pack8(c[qb], 8 * t2);
            }
            __syncthreads();  // P visible to role B
            if (active)
                tr_products(dos, bop);  // dV^T += dO^T P
        } else {
            if (active)
                row_products(dos, c);  // dP
            __syncthreads();
            if (active) {
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg) {
                        const f32x4 dz = *reinterpret_cast<const f32x4 *>(
                            dlt_s + qb * 32 + 8 * rg + 4 * g);
                        const f32x4 pv = *reinterpret_cast<const f32x4 *>(pslot + (qb * 4 + rg) * 256);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            c[qb][4 * rg + e] = pv[e] * (c[qb][4 * rg + e] - dz[e]);
                    }
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int t2 = 0; t2 < 2; ++t2)
                        bop[qb][t2] = pack8(c[qb], 8 * t2);
                tr_products(qs, bop);  // dK^T += Q^T dS
            }
        }
    };

    // The pair of waves of a key group shares one activity decision; every
    // wave reaches the mid-tile barrier.
    auto compute = [&](int t, auto bufc) {
        const int i0 = t * T::BM;
        const bool active = wave_on && i0 <= hi_w && i0 + T::BM - 1 >= lo_w;
        if (wave_full_keys && i0 >= lo_all && i0 + T::BM - 1 <= hi_all)
            body(i0, bufc, IC<0>{}, active);
        else
            body(i0, bufc, IC<1>{}, active);
    };

    issue(t_begin, lds);
    wait_vmem();
    __syncthreads();
    for (int t = t_begin;;) {
        if (t < t_end)
            issue(t + 1, lds + T::STAGE);
        compute(t, IC<0>{});
        wait_vmem();
        __syncthreads();
        if (t == t_end)
            break;
        ++t;
        if (t < t_end)
            issue(t + 1, lds);
        compute(t, IC<1>{});
        wait_vmem();
        __syncthreads();
        if (t == t_end)
            break;
        ++t;
    }

    if (!k_ok)
        return;
    if (!role_a && rope != 0)  // dK with respect to the unrotated keys
        rope_unrotate_acc<DB>(acc, rt, rope_position(b, L, my_k, cu, n_docs, rope), g);
    const float osc = role_a ? 1.0f : scale;
    uint16_t *dst = (role_a ? dV : dK) + base + my_k * rs;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int d = db * 32 + 8 * rg + 4 * g;
            *reinterpret_cast<bf16x4 *>(dst + d) =
                pack4(acc[db][4 * rg] * osc, acc[db][4 * rg + 1] * osc,
                      acc[db][4 * rg + 2] * osc, acc[db][4 * rg + 3] * osc);
        }
}

template __global__ void dkdv_kernel<128>(
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,
    const uint16_t *__restrict__, const float *__restrict__, const float *__restrict__,
    uint16_t *__restrict__, uint16_t *__restrict__, int, int, int, int,
    const int32_t *__restrict__, int, float, float, int, RopeEpi, int);

hipError_t launch_dkdv_paired(const BwdArgs &a, const BwdScalars &s)
{
    using T = KvTile<128>;
    const int nkb = (a.L + T::BN - 1) / T::BN;
    return launch_kernel(dkdv_kernel<128>, dim3(static_cast<unsigned>(nkb * a.B * a.H)),
                         dim3(64 * T::NW), static_cast<hipStream_t>(a.stream), a.Q, a.K, a.V,
                         a.dO, s.lse2, s.delta, a.dK, a.dV, a.B, a.L, a.H, a.causal ? 1 : 0,
                         a.cu, a.n_docs, s.scale_log2, s.scale, nkb, s.rt, s.rope);
}

}  // namespace dd
