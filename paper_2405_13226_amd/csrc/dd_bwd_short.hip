// dd_bwd_short.hip -- the whole attention backward of rows of at most 256
// tokens at D = 64 in one kernel: one workgroup per (b, h) slice.
//
// The slice's Q, dO and K rows are DMA'd into LDS once, and the prologue
// forms delta = rowsum(dO * O) and the LSE in log2 units straight into LDS
// (no workspace).  Each wave owns 32 keys (K and V rows in
// registers, dK and dV accumulators) and walks the 32-query tiles its keys
// are visible to, forming, as the key-resident kernel does,
//   S = Q K^T, P = exp2(S*scale*log2e - lse2), dP - delta (accumulated onto
//   -delta), dS = P (dP - delta), dV^T += dO^T P, dK^T += Q^T dS.
// Every wave then writes its keys' dS of the tile to LDS ([key][query], bf16,
// zeros where it has none; two buffers, alternating by tile), and after a
// barrier two waves form the tile's dQ^T = K^T dS^T over the tile's key range
// (both operands read transposed) while the others go on to the next tile.
// So each input is read from HBM once and S and dP are formed once, where
// the two-kernel backward reads Q, K, V and dO twice and recomputes S and dP
// for dQ; results stay deterministic (no atomics).
#include "dd_bwd.hpp"
#include "dd_launch.hpp"
#include "dd_tile.hpp"

#include <climits>

namespace dd {

// ROWS (64, 128 or 256) is the row capacity: ROWS / 32 waves of 32 keys, and
// LDS for ROWS rows (33, 65 or 130 KiB), so that shorter rows run more
// workgroups per CU.
template <int ROWS>
__global__ void __launch_bounds__(2 * ROWS, 256 / ROWS)
bwd_short_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                 const uint16_t *__restrict__ V, const uint16_t *__restrict__ O,
                 const uint16_t *__restrict__ dO, const float *__restrict__ LSE,
                 uint16_t *__restrict__ dQ, uint16_t *__restrict__ dK,
                 uint16_t *__restrict__ dV, int B, int L, int H, int causal_i,
                 const int32_t *__restrict__ cu, int n_docs, float scale_log2, float scale)
{
    constexpr int D = 64, KK = D / 16, DB = D / 32;
    constexpr int kSNW = ROWS / 32, kSArr = ROWS * D;
    static_assert(kSNW >= DB, "the dQ pass takes DB waves");
    // Q, dO and K rows of the slice, then the dS of two tiles: row = key, the
    // 32 queries of even tiles in columns 0..31 of a D-wide row, odd tiles in
    // 32..63 (so the tile swizzle applies).
    __shared__ __attribute__((aligned(1024))) uint16_t lds[4 * kSArr];
    __shared__ __attribute__((aligned(16))) float rowv[2 * ROWS];  // lse2, -delta
    uint16_t *const qs = lds;
    uint16_t *const dos = lds + kSArr;
    uint16_t *const ks = lds + 2 * kSArr;
    uint16_t *const dss = lds + 3 * kSArr;
    float *const lse_s = rowv;
    float *const ndl_s = rowv + ROWS;

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const int bh = static_cast<int>(blockIdx.x);
    const int b = bh / H, h = bh % H;
    const long long rs = static_cast<long long>(H) * D;
    const long long base = (static_cast<long long>(b) * L * H + h) * D;

    // Q, dO and K rows into LDS; rows past L repeat row L-1.
    {
        DmaPlan<D, ROWS, kSNW> plan;
        plan.init(rs, wave, lane);
        plan.issue(qs, Q + base, rs, 0, L, wave, lane);
        plan.issue(dos, dO + base, rs, 0, L, wave, lane);
        plan.issue(ks, K + base, rs, 0, L, wave, lane);
    }

    // This wave's K and V rows (B operands: column = key); a key past L
    // reads row L-1 (its probabilities are masked to 0, nothing is stored).
    const int my_k = wave * 32 + l32;
    const bool k_ok = my_k < L;
    bf16x8 kf[KK], vf[KK];
    {
        const long long at = base + static_cast<long long>(min(my_k, L - 1)) * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            kf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(K + at + kk * 16));
            vf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(V + at + kk * 16));
        }
    }

    // -delta and lse2 of query wave*32 + l32 (a partial dot product per
    // lane, completed with the lane holding the other half of the row).  A
    // query past L takes row L-1: finite values for rows the mask removes.
    {
        const int q = wave * 32 + l32, qrow = min(q, L - 1);
        const long long at = base + static_cast<long long>(qrow) * rs + g * 8;
        float part = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8 o8 = as_bf16x8(*reinterpret_cast<const u32x4 *>(O + at + kk * 16));
            const bf16x8 d8 = as_bf16x8(*reinterpret_cast<const u32x4 *>(dO + at + kk * 16));
#pragma unroll
            for (int i = 0; i < 8; ++i)
                part += static_cast<float>(o8[i]) * static_cast<float>(d8[i]);
        }
        const float delta = part + __shfl_xor(part, 32);
        if (g == 0) {
            ndl_s[q] = -delta;
            lse_s[q] = LSE[(static_cast<long long>(b) * L + qrow) * H + h] * kLog2e;
        }
    }

    // Allowed queries of this lane's key, and their union / intersection
    // over the wave's keys.
    int qlo_k = 1, qhi_k = 0;
    if (k_ok)
        key_queries(b, L, my_k, causal, cu, n_docs, qlo_k, qhi_k);
    const int lo_w = wave_min(k_ok ? qlo_k : INT_MAX);
    const int hi_w = wave_max(k_ok ? qhi_k : -1);

    int roff[KK], toff[DB][2];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        roff[kk] = tile_off<D>(l32, kk * 16 + g * 8);
    {
        const int G16 = lane >> 4, e = (lane & 15) >> 2, c = lane & 3;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                toff[db][hh] = tile_off<D>(8 * hh + 4 * g + e, db * 32 + 16 * (G16 & 1) + 4 * c);
    }

    f32x16 dk[DB], dv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        dk[db] = f32x16{};
        dv[db] = f32x16{};
    }

    wait_vmem();
    __syncthreads();

    const int nqt = (L + 31) / 32;
    for (int qt = 0; qt < nqt; ++qt) {
        const int i0 = qt * 32;
        // dS of this wave's 32 keys (columns) for the tile's 32 queries (rows
        // 8*rg + 4*g + e of the C layout); zero where the wave has none.
        f32x16 ds = f32x16{};
        if (i0 <= hi_w && i0 + 31 >= lo_w) {
            f32x16 s = f32x16{};
            // dP accumulates onto -delta of its rows.
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const f32x4 nz = *reinterpret_cast<const f32x4 *>(ndl_s + i0 + 8 * rg + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    ds[4 * rg + e] = nz[e];
            }
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int off = i0 * D + roff[kk];
                s = mfma32(lds_row8(qs + off), kf[kk], s);
                ds = mfma32(lds_row8(dos + off), vf[kk], ds);
            }
            const int qlo_r = qlo_k - i0 - 4 * g, qhi_r = qhi_k - i0 - 4 * g;
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const f32x4 lz = *reinterpret_cast<const f32x4 *>(lse_s + i0 + 8 * rg + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 4 * rg + e, qr = 8 * rg + e;
                    float p = fast_exp2(fmaf(s[r], scale_log2, -lz[e]));
                    p = ((qr >= qlo_r) & (qr <= qhi_r)) ? p : 0.f;
                    s[r] = p;
                    ds[r] = p * ds[r];
                }
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const bf16x8 pb = pack8(s, 8 * t2), sb = pack8(ds, 8 * t2);
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const int ro = (i0 + 16 * t2) * D;
                    const bf16x8 ado = join(lds_tr4(dos + ro + toff[db][0]),
                                            lds_tr4(dos + ro + toff[db][1]));
                    const bf16x8 aq = join(lds_tr4(qs + ro + toff[db][0]),
                                           lds_tr4(qs + ro + toff[db][1]));
                    dv[db] = mfma32(ado, pb, dv[db]);
                    dk[db] = mfma32(aq, sb, dk[db]);
                }
            }
        }

        // Even tiles use columns 0..31 of the dS rows, odd tiles 32..63: the
        // buffer written here was last read by the dQ pass of tile qt - 2,
        // which ended before its waves reached the previous tile's barrier.
        const int half = 32 * (qt & 1);
        {
            const int kr = wave * 32 + l32;
#pragma unroll
            for (int rg = 0; rg < 4; ++rg)
                *reinterpret_cast<bf16x4 *>(dss + tile_off<D>(kr, half + 8 * rg + 4 * g)) =
                    pack4(ds[4 * rg], ds[4 * rg + 1], ds[4 * rg + 2], ds[4 * rg + 3]);
        }
        __syncthreads();  // the tile's dS is complete

        // dQ^T (rows db*32.., one block per wave) = K^T dS^T over the keys
        // the tile's queries see (keys of other documents in that range have
        // dS = 0).  The last two waves have the fewest tiles under the causal
        // mask, so they take it.
        if (wave >= kSNW - DB) {
            const int db = wave - (kSNW - DB);
            int klo, khi, tmp;
            query_keys(b, L, i0, causal, cu, n_docs, klo, tmp);
            query_keys(b, L, min(i0 + 31, L - 1), causal, cu, n_docs, tmp, khi);
            const int t0 = half ? toff[1][0] : toff[0][0];
            const int t1 = half ? toff[1][1] : toff[0][1];
            f32x16 acc = f32x16{};
            for (int kb = klo / 16; kb <= khi / 16; ++kb) {
                const uint16_t *kr = ks + kb * 16 * D;
                const uint16_t *sr = dss + kb * 16 * D;
                const bf16x8 a = join(lds_tr4(kr + toff[db][0]), lds_tr4(kr + toff[db][1]));
                const bf16x8 bs = join(lds_tr4(sr + t0), lds_tr4(sr + t1));
                acc = mfma32(a, bs, acc);
            }
            const int q = i0 + l32;
            if (q < L) {
                uint16_t *dQb = dQ + base + static_cast<long long>(q) * rs;
#pragma unroll
                for (int rg = 0; rg < 4; ++rg) {
                    const int d = db * 32 + 8 * rg + 4 * g;
                    *reinterpret_cast<bf16x4 *>(dQb + d) =
                        pack4(acc[4 * rg] * scale, acc[4 * rg + 1] * scale,
                              acc[4 * rg + 2] * scale, acc[4 * rg + 3] * scale);
                }
            }
        }
    }

    // dK (scaled) and dV of this lane's key.
    if (k_ok) {
        uint16_t *dKb = dK + base + static_cast<long long>(my_k) * rs;
        uint16_t *dVb = dV + base + static_cast<long long>(my_k) * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const int d = db * 32 + 8 * rg + 4 * g;
                *reinterpret_cast<bf16x4 *>(dKb + d) =
                    pack4(dk[db][4 * rg] * scale, dk[db][4 * rg + 1] * scale,
                          dk[db][4 * rg + 2] * scale, dk[db][4 * rg + 3] * scale);
                *reinterpret_cast<bf16x4 *>(dVb + d) = pack4(
                    dv[db][4 * rg], dv[db][4 * rg + 1], dv[db][4 * rg + 2], dv[db][4 * rg + 3]);
            }
    }
}

hipError_t launch_bwd_short(const BwdArgs &a, const BwdScalars &s)
{
    const auto kern = a.L <= 64 ? bwd_short_kernel<64>
                      : a.L <= 128 ? bwd_short_kernel<128> : bwd_short_kernel<256>;
    const int rows = a.L <= 64 ? 64 : a.L <= 128 ? 128 : 256;
    return launch_kernel(kern, dim3(static_cast<unsigned>(a.B * a.H)), dim3(2 * rows),
                         static_cast<hipStream_t>(a.stream), a.Q, a.K, a.V, a.O, a.dO, a.LSE,
                         a.dQ, a.dK, a.dV, a.B, a.L, a.H, a.causal ? 1 : 0, a.cu, a.n_docs,
                         s.scale_log2, s.scale);
}

}  // namespace dd
