// dd_bwd.hip -- backward of masked causal attention on gfx950, recomputing
// the probabilities from the forward's log-sum-exp.
//
// Two launches on the caller's stream:
//   1. dq:    query-resident.  One workgroup = 4 waves = 128 queries; each
//             wave keeps its queries' Q and dO rows in registers.  It first
//             forms delta_i = sum_d dO_id O_id and the LSE in log2 units for
//             its queries and writes -delta and the LSE, fp32, to a [B*H][L]
//             workspace (one contiguous row per (b, h)); then it walks the key tiles (64
//             keys) its queries see and forms
//               S^T = K Q^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T,
//             with K and V tiles in LDS (K^T read transposed).
//   2. dkdv:  key-resident, 128 keys per workgroup.  For D = 128
//             (dd_dkdv.hip) the two waves of a 32-key group keep K (one) and
//             V (the other) rows in registers; for D = 64 (here) one wave
//             holds both.  They walk the query tiles (64 queries) their keys
//             are visible to and form
//               S = Q K^T, P = exp2(S*scale*log2e - lse2),
//               dP - delta = dO V^T accumulated onto -delta,  dS = P (dP - delta),
//               dV^T += dO^T P,  dK^T += Q^T dS,
//             reading lse2 and -delta of each tile from the workspace.
//             Q and dO tiles arrive row-major in LDS by direct DMA; S and dP
//             read them row-wise, dV^T and dK^T transposed (ds_read_b64_tr_b16).
// Splitting dQ from dK/dV keeps every output owned by exactly one workgroup:
// no atomics, deterministic results, at the cost of recomputing S and dP.
// At D = 64, rows of at most 256 tokens without RoPE instead take one launch
// (dd_bwd_short.hip) in which a slice fits one workgroup and S and dP are
// formed once.
#include "dd_bwd.hpp"
#include "dd_tile.hpp"
#include "dd_launch.hpp"
#include "dd_prof.hpp"
#include "dd_attn.h"

namespace dd {

// ---------------------------------------------------------------------------
// 1. dK, dV
// ---------------------------------------------------------------------------

// Key-resident dK/dV for small head dims: one wave owns the 32 keys of a
// group with both K and V in registers and both accumulators, and walks the
// 64-query tile as two 32-query halves to keep its live registers low enough
// for several waves per SIMD.
//
// PERSIST = false: one work item (key block) per workgroup.  PERSIST = true:
// a workgroup walks its work items (item_bid) back to back; during an
// item's last query tile it loads the next item's first Q/dO tile into the
// free LDS stage, and after that tile the next item's K and V rows (holding
// them during the tile as well would spill at D = 64).
template <int D>
struct KvTile1 {
    static constexpr int BN = 128;            // keys per workgroup
    static constexpr int BM = 64;             // queries per tile
    static constexpr int NW = 4;
    static constexpr int TILE = BM * D;
    static constexpr int STAGE = 2 * TILE + 2 * BM * 2;
};

template <int D, bool PERSIST>
__global__ void __launch_bounds__(256, 2)
dkdv1_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
             const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
             const float *__restrict__ lse2g, const float *__restrict__ ndeltag,
             uint16_t *__restrict__ dK, uint16_t *__restrict__ dV, int B, int L, int H,
             int causal_i, const int32_t *__restrict__ cu, int n_docs, float scale_log2,
             float scale, int nkb, RopeEpi rt, int rope)
{
    using T = KvTile1<D>;
    constexpr int KK = D / 16;
    constexpr int DB = D / 32;
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * T::STAGE];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const long long rs = static_cast<long long>(H) * D;
    const int n_items = nkb * B * H;
    const int G = static_cast<int>(gridDim.x);

    int k_item = 0;
    const int bid = item_bid(0, static_cast<int>(blockIdx.x), G, n_items);
    if (bid < 0)
        return;
    KvItem it = kv_item<D, T>(bid, nkb, B, L, H, causal, cu, n_docs), nit = it;

    // Per-lane state of the current item.
    int my_k, qlo_k, qhi_k, lo_w, hi_w, lo_all, hi_all;
    bool k_ok, wave_on, wave_full_keys;
    auto setup = [&](const KvItem &x) __attribute__((always_inline)) {
        const int k0w = x.kvb * T::BN + wave * 32;
        my_k = k0w + l32;
        k_ok = my_k < L;
        qlo_k = 1;
        qhi_k = 0;
        if (k_ok)
            key_queries(x.b, L, my_k, causal, cu, n_docs, qlo_k, qhi_k);
        wave_on = k0w < L;
        lo_w = wave_min(k_ok ? qlo_k : 0x7fffffff);
        hi_w = wave_max(k_ok ? qhi_k : -1);
        lo_all = wave_max(k_ok ? qlo_k : -1);
        hi_all = wave_min(k_ok ? qhi_k : 0x7fffffff);
        wave_full_keys = (k0w + 31) < L;
    };

    // K and V rows of this lane's key (B operands: column = key).  A key past
    // L reads row L-1 instead (no branch around the loads, so they stay in
    // flight until needed): its probabilities are masked to exactly 0 by a
    // select, and its dK/dV column is never stored.
    bf16x8 kf[KK], vf[KK];
    auto load_kv = [&](const KvItem &x) __attribute__((always_inline)) {
        const int key = min(x.kvb * T::BN + wave * 32 + l32, L - 1);
        const long long at = x.base + key * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            kf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(K + at + kk * 16));
            vf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(V + at + kk * 16));
        }
    };

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
    // kDmaAsm lets the compiler spill the one-block form (28 VGPRs).
    DmaPlan<D, T::BM, T::NW, kDmaAsmCast> plan;
    plan.init(rs, wave, lane);

    auto body = [&](int i0, auto bufc, auto maskc) {
        constexpr int BUF = decltype(bufc)::value;
        constexpr bool MASKED = decltype(maskc)::value != 0;
        const uint16_t *qs = lds + BUF * T::STAGE;
        const uint16_t *dos = qs + T::TILE;
        const float *lse_s = reinterpret_cast<const float *>(qs + 2 * T::TILE);
        const float *ndl_s = lse_s + T::BM;
        const int qlo_r = qlo_k - i0 - 4 * g, qhi_r = qhi_k - i0 - 4 * g;
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            // A boundary tile's half whose queries none of the wave's keys
            // sees adds nothing (its probabilities are all 0): skipped.
            if (MASKED && (i0 + 32 * qb > hi_w || i0 + 32 * qb + 31 < lo_w))
                continue;
            // dP accumulates onto -delta of its rows (C layout: register
            // 4*rg + e holds query 8*rg + 4*g + e), so the products give
            // dP - delta directly.
            f32x16 s = f32x16{}, dp;
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const f32x4 nz = *reinterpret_cast<const f32x4 *>(ndl_s + qb * 32 + 8 * rg + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    dp[4 * rg + e] = nz[e];
            }
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int off = qb * 32 * D + roff[kk];
                s = mfma32(lds_row8(qs + off), kf[kk], s);
                dp = mfma32(lds_row8(dos + off), vf[kk], dp);
            }
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) {
                const int ql = qb * 32 + 8 * rg + 4 * g;
                const f32x4 lz = *reinterpret_cast<const f32x4 *>(lse_s + ql);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 4 * rg + e;
                    float p = fast_exp2(fmaf(s[r], scale_log2, -lz[e]));
                    if constexpr (MASKED) {
                        const int qr = qb * 32 + 8 * rg + e;
                        const bool ok = (qr >= qlo_r) & (qr <= qhi_r);
                        p = ok ? p : 0.f;
                    }
                    s[r] = p;
                    dp[r] = p * dp[r];
                }
            }
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const bf16x8 pb = pack8(s, 8 * t2), sb = pack8(dp, 8 * t2);
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const int ro = (qb * 32 + 16 * t2) * D;
                    const bf16x8 ado = join(lds_tr4(dos + ro + toff[db][0]),
                                            lds_tr4(dos + ro + toff[db][1]));
                    const bf16x8 aq = join(lds_tr4(qs + ro + toff[db][0]),
                                           lds_tr4(qs + ro + toff[db][1]));
                    dv[db] = mfma32(ado, pb, dv[db]);
                    dk[db] = mfma32(aq, sb, dk[db]);
                }
            }
        }
    };

    auto compute = [&](int t, auto bufc) {
        const int i0 = t * T::BM;
        if (!(wave_on && i0 <= hi_w && i0 + T::BM - 1 >= lo_w))
            return;
        if (wave_full_keys && i0 >= lo_all && i0 + T::BM - 1 <= hi_all)
            body(i0, bufc, IC<0>{});
        else
            body(i0, bufc, IC<1>{});
    };

    // dK (scaled, and with respect to the unrotated keys under RoPE) and dV
    // of the current item.
    auto store = [&]() __attribute__((always_inline)) {
        if (k_ok && rope != 0) {
            // Keeps the frequency arithmetic here: hoisted out of the item
            // loop it would hold registers across every tile.
            int gl = g;
            asm volatile("" : "+v"(gl));
            rope_unrotate_acc<DB>(dk, rt, rope_position(it.b, L, my_k, cu, n_docs, rope), gl);
        }
        // Every lane takes part in the store's lane exchange.
        const long long row = k_ok ? my_k : 0;
        uint16_t *dKb = dK + it.base + row * rs;
        uint16_t *dVb = dV + it.base + row * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            store_block_bf16(dKb + db * 32, dk[db], scale, g, k_ok);
            store_block_bf16(dVb + db * 32, dv[db], 1.0f, g, k_ok);
        }
    };

    setup(it);
    load_kv(it);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        dk[db] = f32x16{};
        dv[db] = f32x16{};
    }
    int t = it.t_begin;
    kv_issue<D, T>(plan, lds, Q, dO, lse2g, ndeltag, it, t, L, rs, wave, lane);
    wait_vmem();
    __syncthreads();

    // One query tile in LDS stage BUF; the next tile (of this item or the
    // next one) goes to the other stage.  Returns false after the last item.
    auto step = [&](auto bufc) __attribute__((always_inline)) -> bool {
        constexpr int BUF = decltype(bufc)::value;
        uint16_t *other = lds + (1 - BUF) * T::STAGE;
        const bool last = t == it.t_end;
        bool more = false;
        if (!last) {
            kv_issue<D, T>(plan, other, Q, dO, lse2g, ndeltag, it, t + 1, L, rs, wave, lane);
        } else if constexpr (PERSIST) {
            const int nbid = item_bid(k_item + 1, static_cast<int>(blockIdx.x), G, n_items);
            more = nbid >= 0;
            if (more) {
                nit = kv_item<D, T>(nbid, nkb, B, L, H, causal, cu, n_docs);
                kv_issue<D, T>(plan, other, Q, dO, lse2g, ndeltag, nit, nit.t_begin, L, rs, wave,
                               lane);
            }
        }
        compute(t, bufc);
        if (more)  // K and V of the next item (registers free after the tile)
            load_kv(nit);
        wait_vmem();
        __syncthreads();
        if (!last) {
            ++t;
            return true;
        }
        store();
        if (!PERSIST || !more)
            return false;
        ++k_item;
        it = nit;
        setup(it);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            dk[db] = f32x16{};
            dv[db] = f32x16{};
        }
        t = it.t_begin;
        return true;
    };
    for (;;) {
        if (!step(IC<0>{}))
            break;
        if (!step(IC<1>{}))
            break;
    }
}

// ---------------------------------------------------------------------------
// 2. dQ, delta and log2-LSE
// ---------------------------------------------------------------------------
template <int D>
struct QTile {
    static constexpr int BM = 128;         // queries per workgroup
    static constexpr int BN = 64;          // keys per tile
    static constexpr int TILE = BN * D;    // elements of a K or V tile
    static constexpr int STAGE = 2 * TILE; // K then V
};

// Row lengths (tokens) up to which dQ runs persistently (D = 64); as for
// dK/dV the test ignores document masking.
constexpr long long kDqPersistMaxSpan = 2048;

// A query-block work item of the dQ kernel: one block of QTile::BM queries
// of one (b, h) slice and the key tiles those queries see.
struct QItem {
    int b, bh, qb, t_begin, t_end;
    long long base;  // element offset of (b, row 0, h, 0)
};

template <int D>
__device__ __forceinline__ QItem q_item(int bid, int nqb, int B, int L, int H, bool causal,
                                        const int32_t *__restrict__ cu, int n_docs)
{
    using T = QTile<D>;
    QItem it;
    int jb;
    block_slice(bid, nqb, B * H, it.bh, jb);
    it.qb = nqb - 1 - jb;  // the last query blocks see the most keys: first
    it.b = it.bh / H;
    it.base = (static_cast<long long>(it.b) * L * H + it.bh % H) * D;
    const int qf0 = it.qb * T::BM, ql = min(qf0 + T::BM - 1, L - 1);
    int wlo, whi, tmp;
    query_keys(it.b, L, qf0, causal, cu, n_docs, wlo, tmp);
    query_keys(it.b, L, ql, causal, cu, n_docs, tmp, whi);
    it.t_begin = wlo / T::BN;
    it.t_end = whi / T::BN;
    return it;
}

// PERSIST = false: one query block per workgroup.  PERSIST = true (short
// rows, D = 64 only; at D = 128 the item loop spills): a workgroup walks
// its query blocks in the order of item_bid; during a block's last key tile
// it DMAs the next block's first K/V tile into the free stage and the next
// block's Q and dO rows into LDS areas of their own (read into registers
// after that tile), and loads its O rows and LSE into registers.
// Waves per SIMD: four in the one-block D = 64 form (at most 128 VGPRs),
// two otherwise (the persistent form's item loop and D = 128 need more).
template <int D, bool PERSIST>
__global__ void __launch_bounds__(256, (D == 64 && !PERSIST) ? 4 : 2)
dq_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
          const uint16_t *__restrict__ V, const uint16_t *__restrict__ O,
          const uint16_t *__restrict__ dO, const float *__restrict__ LSE,
          float *__restrict__ lse2g, float *__restrict__ ndeltag,
          uint16_t *__restrict__ dQ, int B, int L, int H, int causal_i,
          const int32_t *__restrict__ cu, int n_docs, float scale_log2, float scale, int nqb,
          RopeEpi rt, int rope)
{
    using T = QTile<D>;
    constexpr int KK = D / 16;
    constexpr int DB = D / 32;
    // Persistent (D = 64): the next item's Q and dO rows are staged here by
    // direct loads during the current item's last tile, its O rows and LSE
    // loaded into registers at the same time.
    constexpr bool kRowStage = PERSIST;
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * T::STAGE + (kRowStage ? 2 * T::BM * D : 0)];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const long long rs = static_cast<long long>(H) * D;
    const int n_items = nqb * B * H;
    const int G = static_cast<int>(gridDim.x);

    int k_item = 0;
    const int bid = item_bid(0, static_cast<int>(blockIdx.x), G, n_items);
    if (bid < 0)
        return;
    QItem it = q_item<D>(bid, nqb, B, L, H, causal, cu, n_docs), nit = it;

    // Per-lane state of the current item.
    int my_q, lo_q, hi_q, lo_w, hi_w, lo_all, hi_all;
    bool q_ok, wave_on, wave_full_rows;
    auto setup = [&](const QItem &x) __attribute__((always_inline)) {
        const int q0w = x.qb * T::BM + wave * 32;
        my_q = q0w + l32;
        q_ok = my_q < L;
        lo_q = 1;
        hi_q = 0;
        if (q_ok)
            query_keys(x.b, L, my_q, causal, cu, n_docs, lo_q, hi_q);
        wave_on = q0w < L;
        lo_w = wave_min(q_ok ? lo_q : 0x7fffffff);
        hi_w = wave_max(q_ok ? hi_q : -1);
        lo_all = wave_max(q_ok ? lo_q : -1);
        hi_all = wave_min(q_ok ? hi_q : 0x7fffffff);
        wave_full_rows = (q0w + 31) < L;
    };

    // Q, dO and O rows of this lane's query (k-slots 8g..8g+7 of each
    // 16-wide step; load_rows), then delta = rowsum(dO * O): a partial per
    // lane, completed with the lane holding the other half of the row; -delta
    // and the LSE in log2 units are written, in [B*H][L] rows, for the dK/dV
    // kernel that runs after this one (finish_rows).  A query past L reads
    // row L-1 instead (its probabilities are masked to exactly 0 by a select
    // and nothing of it is stored).
    bf16x8 qf[KK], dof[KK], of[KK];
    float neg_lse2 = 0.f, my_delta = 0.f, lse_in = 0.f;
    // O rows and the LSE of this lane's query (for delta and lse2).
    auto load_o = [&](const QItem &x) __attribute__((always_inline)) {
        const int qrow = min(x.qb * T::BM + wave * 32 + l32, L - 1);
        const long long at = x.base + qrow * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            of[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(O + at + kk * 16));
        lse_in = LSE[(static_cast<long long>(x.b) * L + qrow) * H + x.bh % H];
    };
    auto load_rows = [&](const QItem &x) __attribute__((always_inline)) {
        const int qrow = min(x.qb * T::BM + wave * 32 + l32, L - 1);
        const long long at = x.base + qrow * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(Q + at + kk * 16));
            dof[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(dO + at + kk * 16));
        }
        load_o(x);
    };
    auto finish_rows = [&](const QItem &x) __attribute__((always_inline)) {
        const int q = x.qb * T::BM + wave * 32 + l32;
        float part = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                part += static_cast<float>(of[kk][i]) * static_cast<float>(dof[kk][i]);
        my_delta = part + __shfl_xor(part, 32);
        const float lse2 = lse_in * kLog2e;
        neg_lse2 = -lse2;
        if (q < L && g == 0) {
            const long long wrow = static_cast<long long>(x.bh) * L;
            ndeltag[wrow + q] = -my_delta;
            lse2g[wrow + q] = lse2;
        }
    };

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

    f32x16 dq[DB];
    DmaPlan<D, T::BN, 4, kDmaAsm> plan;
    plan.init(rs, wave, lane);
    auto issue = [&](const QItem &x, int t, uint16_t *stage) __attribute__((always_inline)) {
        plan.issue(stage, K + x.base, rs, t * T::BN, L, wave, lane);
        plan.issue(stage + T::TILE, V + x.base, rs, t * T::BN, L, wave, lane);
    };

    // One tile; MASKED selects the boundary-tile variant at compile time.
    auto body = [&](int j0, auto bufc, auto maskc) {
        constexpr int BUF = decltype(bufc)::value;
        constexpr bool MASKED = decltype(maskc)::value != 0;
        const uint16_t *ks = lds + BUF * T::STAGE;
        const uint16_t *vs = ks + T::TILE;

        // Per 32-key block: S^T = K Q^T and dP^T = V dO^T (column = this
        // lane's query), dS^T, then dQ^T += K^T dS^T with K^T read transposed.
        // Blocks are processed one after the other so that only one block's
        // scores are live, which leaves registers for LDS reads in flight.
        const int lo_r = lo_q - j0 - 4 * g, hi_r = hi_q - j0 - 4 * g;
        if constexpr (!MASKED && PERSIST) {
            // Full tiles of the persistent form (two waves per SIMD anyway,
            // its item loop holds more registers): both blocks' products at
            // once (four independent accumulator chains), then both blocks'
            // dS, then dQ.  In the other form the extra registers would cost
            // the third wave per SIMD, which is worth more.
            float nd = -my_delta;
            asm volatile("" : "+v"(nd));
            f32x16 s2[2], dp2[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                s2[kb] = f32x16{};
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    dp2[kb][r] = nd;
            }
#pragma unroll
            for (int k0 = 0; k0 < KK; k0 += 2) {
                bf16x8 ka[2][2], va[2][2];
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        const int off = kb * 32 * D + roff[k0 + i];
                        ka[kb][i] = lds_row8(ks + off);
                        va[kb][i] = lds_row8(vs + off);
                    }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb) {
                        s2[kb] = mfma32(ka[kb][i], qf[k0 + i], s2[kb]);
                        dp2[kb] = mfma32(va[kb][i], dof[k0 + i], dp2[kb]);
                    }
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    dp2[kb][r] = fast_exp2(fmaf(s2[kb][r], scale_log2, neg_lse2)) * dp2[kb][r];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                bf16x8 kt[2][DB];
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                    for (int db = 0; db < DB; ++db) {
                        const uint16_t *kr = ks + (kb * 32 + 16 * t2) * D;
                        kt[t2][db] = join(lds_tr4(kr + toff[db][0]), lds_tr4(kr + toff[db][1]));
                    }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2) {
                    const bf16x8 sb = pack8(dp2[kb], 8 * t2);
#pragma unroll
                    for (int db = 0; db < DB; ++db)
                        dq[db] = mfma32(kt[t2][db], sb, dq[db]);
                }
            }
            return;
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            // A boundary tile's 32-key block that none of the wave's queries
            // sees adds nothing (its probabilities are all 0): skipped.
            if (MASKED && (j0 + 32 * kb > hi_w || j0 + 32 * kb + 31 < lo_w))
                continue;
            // The A fragments are read in batches of KB_STEP k-steps before
            // their products, so several LDS reads are in flight at once; in
            // the one-block D = 64 form one k-step at a time keeps the kernel
            // within 128 VGPRs, four waves per SIMD.
            constexpr int KB_STEP = KK >= 8 ? 4 : (PERSIST ? 2 : 1);
            // dP^T accumulates onto -delta (this lane's query), so the
            // products give dP - delta, and the fill runs beside the S
            // products instead of a subtraction after them.  The opaque copy
            // keeps the compiler from hoisting the filled registers out of
            // the tile loop.
            float nd = -my_delta;
            asm volatile("" : "+v"(nd));
            f32x16 s = f32x16{}, dp;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                dp[r] = nd;
#pragma unroll
            for (int k0 = 0; k0 < KK; k0 += KB_STEP) {
                bf16x8 ka[KB_STEP], va[KB_STEP];
#pragma unroll
                for (int i = 0; i < KB_STEP; ++i) {
                    const int off = kb * 32 * D + roff[k0 + i];
                    ka[i] = lds_row8(ks + off);
                    va[i] = lds_row8(vs + off);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < KB_STEP; ++i) {
                    s = mfma32(ka[i], qf[k0 + i], s);
                    dp = mfma32(va[i], dof[k0 + i], dp);
                }
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float p = fast_exp2(fmaf(s[r], scale_log2, neg_lse2));
                if constexpr (MASKED) {
                    const int kr = kb * 32 + 8 * (r >> 2) + (r & 3);
                    const bool ok = (kr >= lo_r) & (kr <= hi_r);
                    p = ok ? p : 0.f;
                }
                dp[r] = p * dp[r];
            }
            bf16x8 kt[2][DB];
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const uint16_t *kr = ks + (kb * 32 + 16 * t2) * D;
                    kt[t2][db] = join(lds_tr4(kr + toff[db][0]), lds_tr4(kr + toff[db][1]));
                }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const bf16x8 sb = pack8(dp, 8 * t2);
#pragma unroll
                for (int db = 0; db < DB; ++db)
                    dq[db] = mfma32(kt[t2][db], sb, dq[db]);
            }
        }
    };

    auto compute = [&](int t, auto bufc) {
        const int j0 = t * T::BN;
        if (!(wave_on && j0 <= hi_w && j0 + T::BN - 1 >= lo_w))
            return;
        if (wave_full_rows && j0 >= lo_all && j0 + T::BN - 1 <= hi_all)
            body(j0, bufc, IC<0>{});
        else
            body(j0, bufc, IC<1>{});
    };

    // dQ (scaled, and with respect to the unrotated queries under RoPE) of
    // the current item.
    auto store = [&]() __attribute__((always_inline)) {
        if (q_ok && rope != 0) {
            // Keeps the frequency arithmetic here: hoisted out of the item
            // loop it would hold registers across every tile.
            int gl = g;
            RopeEpi r = rt;
            asm volatile("" : "+v"(gl), "+s"(r.p0), "+s"(r.p1), "+s"(r.p2), "+s"(r.p3),
                         "+s"(r.r4), "+s"(r.r16));
            rope_unrotate_acc<DB>(dq, r, rope_position(it.b, L, my_q, cu, n_docs, rope), gl);
        }
        // Every lane takes part in the store's lane exchange.
        uint16_t *dQb = dQ + it.base + static_cast<long long>(q_ok ? my_q : 0) * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db)
            store_block_bf16(dQb + db * 32, dq[db], scale, g, q_ok);
    };

    setup(it);
    load_rows(it);
    finish_rows(it);
#pragma unroll
    for (int db = 0; db < DB; ++db)
        dq[db] = f32x16{};
    int t = it.t_begin;
    issue(it, t, lds);
    wait_vmem();
    __syncthreads();

    // One key tile in LDS stage BUF; the next tile (of this item or the next
    // one) goes to the other stage.  Returns false after the last item.
    auto step = [&](auto bufc) __attribute__((always_inline)) -> bool {
        constexpr int BUF = decltype(bufc)::value;
        uint16_t *other = lds + (1 - BUF) * T::STAGE;
        const bool last = t == it.t_end;
        bool more = false;
        if (!last) {
            issue(it, t + 1, other);
        } else if constexpr (PERSIST) {
            const int nbid = item_bid(k_item + 1, static_cast<int>(blockIdx.x), G, n_items);
            more = nbid >= 0;
            if (more) {
                nit = q_item<D>(nbid, nqb, B, L, H, causal, cu, n_docs);
                issue(nit, nit.t_begin, other);
                if constexpr (kRowStage) {  // 64-row halves with the tile plan
                    uint16_t *rows = lds + 2 * T::STAGE;
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2) {
                        const int r0 = nit.qb * T::BM + h2 * T::BN;
                        plan.issue(rows + h2 * T::BN * D, Q + nit.base, rs, r0, L, wave, lane);
                        plan.issue(rows + T::BM * D + h2 * T::BN * D, dO + nit.base, rs, r0, L,
                                   wave, lane);
                    }
                    load_o(nit);  // registers free since the item's start
                }
            }
        }
        compute(t, bufc);
        if (!kRowStage && more)  // Q, dO, O rows of the next item (registers free after the tile)
            load_rows(nit);
        wait_vmem();
        __syncthreads();
        if (kRowStage && more) {  // the staged rows are in LDS
            const uint16_t *rows = lds + 2 * T::STAGE + wave * 32 * D;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                qf[kk] = lds_row8(rows + roff[kk]);
                dof[kk] = lds_row8(rows + T::BM * D + roff[kk]);
            }
            // Every wave has its rows before the next item's last tile
            // stages the following rows (a one-tile item has no other
            // barrier in between).
            __syncthreads();
        }
        if (!last) {
            ++t;
            return true;
        }
        if constexpr (!PERSIST) {
            return false;  // stored after the loop
        } else {
            store();
            if (!more)
                return false;
        }
        ++k_item;
        it = nit;
        setup(it);
        finish_rows(it);
#pragma unroll
        for (int db = 0; db < DB; ++db)
            dq[db] = f32x16{};
        t = it.t_begin;
        return true;
    };
    for (;;) {
        if (!step(IC<0>{}))
            break;
        if (!step(IC<1>{}))
            break;
    }
    if constexpr (!PERSIST)
        store();
}

// Explicit instantiations: the host-side launch stubs of these kernel
// templates are emitted here unconditionally (clang's host pass does not
// always emit them for templates only referenced through a function pointer).
#define DD_KV_ARGS                                                                               \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        const uint16_t *__restrict__, const float *__restrict__, const float *__restrict__,      \
        uint16_t *__restrict__, uint16_t *__restrict__, int, int, int, int,                      \
        const int32_t *__restrict__, int, float, float, int, RopeEpi, int
#define DD_Q_ARGS                                                                                \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        const uint16_t *__restrict__, const uint16_t *__restrict__, const float *__restrict__,   \
        float *__restrict__, float *__restrict__, uint16_t *__restrict__, int, int, int, int,     \
        const int32_t *__restrict__, int, float, float, int, RopeEpi, int
template __global__ void dkdv1_kernel<64, false>(DD_KV_ARGS);  // D = 64: single-role waves
template __global__ void dkdv1_kernel<64, true>(DD_KV_ARGS);
template __global__ void dq_kernel<64, false>(DD_Q_ARGS);
template __global__ void dq_kernel<64, true>(DD_Q_ARGS);
template __global__ void dq_kernel<128, false>(DD_Q_ARGS);  // D = 128: never persistent
#undef DD_KV_ARGS
#undef DD_Q_ARGS

// ---------------------------------------------------------------------------
template <int D>
static int launch_bwd_d(const BwdArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const size_t region = align256(static_cast<size_t>(a.B) * a.H * a.L * sizeof(float));
    float *lse2 = static_cast<float *>(a.workspace);
    float *ndelta = reinterpret_cast<float *>(static_cast<char *>(a.workspace) + region);
    BwdScalars s;
    s.lse2 = lse2;
    s.ndelta = ndelta;
    s.scale = 1.0f / sqrtf(static_cast<float>(D));
    s.scale_log2 = s.scale * kLog2e;
    // RoPE: 0 off, 1 row positions, 2 document-local positions.
    s.rope = a.rope_base > 0.0 ? (a.rope_doc && a.cu ? 2 : 1) : 0;
    s.rt = s.rope ? rope_epi(a.rope_base, D) : RopeEpi{};

    hipError_t e;
    if constexpr (D == 64)
        if (a.L <= kShortMaxRow && s.rope == 0) {
            ProfScope prof(K_BWD_SHORT, st);
            e = launch_bwd_short(a, s);
            return e == hipSuccess ? DD_OK : DD_ERR_HIP;
        }

    // dQ first: it also writes -delta and log2-LSE, which dK/dV reads.
    const int nqb = (a.L + QTile<D>::BM - 1) / QTile<D>::BM;
    {
        const long long all =
            (static_cast<long long>(nqb) * a.B * a.H + kXcds - 1) / kXcds * kXcds;
        // Persistent only at D = 64: at D = 128 its item loop spills.
        long long pgrid = 0;
        if constexpr (D == 64)
            if (a.L <= kDqPersistMaxSpan)
                pgrid = persistent_grid<dq_kernel<D, true>>(256);
        const bool persist = pgrid > 0 && pgrid < all;
        auto kern = dq_kernel<D, false>;
        if constexpr (D == 64)
            if (persist)
                kern = dq_kernel<D, true>;
        ProfScope prof(K_DQ, st);
        e = launch_kernel(kern,
                          dim3(static_cast<unsigned>(persist ? pgrid : all)), dim3(256), st, a.Q,
                          a.K, a.V, a.O, a.dO, a.LSE, lse2, ndelta, a.dQ, a.B, a.L, a.H,
                          a.causal ? 1 : 0, a.cu, a.n_docs, s.scale_log2, s.scale, nqb, s.rt,
                          s.rope);
    }
    if (e != hipSuccess)
        return DD_ERR_HIP;

    {
        ProfScope prof(K_DKDV, st);
        if constexpr (D == 64) {
            using T = KvTile1<D>;
            const int nkb = (a.L + T::BN - 1) / T::BN;
            const long long n_items = static_cast<long long>(nkb) * a.B * a.H;
            const long long all = (n_items + kXcds - 1) / kXcds * kXcds;
            // Persistent for short rows, as many workgroups as are resident
            // at once (two per CU).
            const long long pgrid = a.L <= kPersistMaxSpan
                                        ? persistent_grid<dkdv1_kernel<D, true>>(64 * T::NW)
                                        : 0;
            const bool persist = pgrid > 0 && pgrid < all;
            auto kern = persist ? dkdv1_kernel<D, true> : dkdv1_kernel<D, false>;
            const long long grid = persist ? pgrid : all;
            e = launch_kernel(kern, dim3(static_cast<unsigned>(grid)), dim3(64 * T::NW), st, a.Q,
                              a.K, a.V, a.dO, lse2, ndelta, a.dK, a.dV, a.B, a.L, a.H,
                              a.causal ? 1 : 0, a.cu, a.n_docs, s.scale_log2, s.scale, nkb, s.rt,
                              s.rope);
        } else {
            e = launch_dkdv_paired(a, s);
        }
    }
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_bwd(const BwdArgs &a)
{
    return a.D == 64 ? launch_bwd_d<64>(a) : launch_bwd_d<128>(a);
}

}  // namespace dd
