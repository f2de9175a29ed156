// dd_bwd.hpp -- pieces of the attention backward shared by its translation
// units (dd_bwd.hip: dK/dV for D = 64, dQ and the launcher;
// dd_dkdv.hip: dK/dV for D = 128; dd_bwd_short.hip: the one-kernel backward
// of short rows at D = 64).
#pragma once

#include "dd_device.hpp"
#include "dd_internal.h"
#include "dd_rope.hpp"
#include "dd_tile.hpp"


namespace dd {

// Per-call values every backward kernel takes, derived once by the launcher.
struct BwdScalars {
    const float *lse2;   // [B*H][L] log-sum-exp in log2 units (workspace)
    const float *ndelta; // [B*H][L] -rowsum(dO * O) (workspace)
    float scale_log2;    // softmax scale times log2(e)
    float scale;         // softmax scale 1/sqrt(D)
    RopeEpi rt;          // rotary frequencies for the dQ / dK epilogues
    int rope;            // 0 off, 1 row positions, 2 document-local positions
};

// dK and dV for D = 128 with the paired-wave kernel (dd_dkdv.hip); returns the
// runtime's launch status.
hipError_t launch_dkdv_paired(const BwdArgs &a, const BwdScalars &s);

// Rows of at most this many tokens at D = 64 (without RoPE) take the one-kernel
// backward of dd_bwd_short.hip: one workgroup per (b, h) slice.
constexpr int kShortMaxRow = 256;
hipError_t launch_bwd_short(const BwdArgs &a, const BwdScalars &s);

// Rows of at most this many tokens take the persistent dK/dV forms: a key
// block then visits few query tiles, and a workgroup that walks its blocks
// back to back hides each block's set-up behind the previous one; longer
// rows have long items and run one item per workgroup (hardware dispatch).
// The test is on the row length even under document masking: documents make
// the work per block uneven, which the hardware's dispatch balances and the
// persistent forms' fixed order does not.
constexpr long long kPersistMaxSpan = 1024;

// ---------------------------------------------------------------------------
// Work items of the persistent dK/dV kernels
// ---------------------------------------------------------------------------

// A work item: one key block of one (b, h) slice and the query tiles its
// keys are visible to.
struct KvItem {
    int b, bh, kvb, t_begin, t_end;
    long long base;  // element offset of (b, row 0, h, 0)
};

// Tile shape T: T::BN keys per item, T::BM queries per tile.
template <int D, class T>
__device__ __forceinline__ KvItem kv_item(int bid, int nkb, int B, int L, int H, bool causal,
                                          const int32_t *__restrict__ cu, int n_docs)
{
    KvItem it;
    block_slice(bid, nkb, B * H, it.bh, it.kvb);
    it.b = it.bh / H;
    it.base = (static_cast<long long>(it.b) * L * H + it.bh % H) * D;
    const int kf0 = it.kvb * T::BN, kl = min(kf0 + T::BN - 1, L - 1);
    int wlo, whi, tmp;
    key_queries(it.b, L, kf0, causal, cu, n_docs, wlo, tmp);
    key_queries(it.b, L, kl, causal, cu, n_docs, tmp, whi);
    it.t_begin = wlo / T::BM;
    it.t_end = whi / T::BM;
    return it;
}

// Direct-to-LDS loads of query tile t of item x into `stage`: the Q and dO
// tiles (T::TILE elements each), then lse2 and -delta of its rows (waves 0
// and 1).
template <int D, class T, int MODE>
__device__ __forceinline__ void kv_issue(const DmaPlan<D, T::BM, T::NW, MODE> &plan, uint16_t *stage,
                                         const uint16_t *__restrict__ Q,
                                         const uint16_t *__restrict__ dO,
                                         const float *__restrict__ lse2g,
                                         const float *__restrict__ ndeltag, const KvItem &x, int t,
                                         int L, long long rs, int wave, int lane)
{
    const int i0 = t * T::BM;
    plan.issue(stage, Q + x.base, rs, i0, L, wave, lane);
    plan.issue(stage + T::TILE, dO + x.base, rs, i0, L, wave, lane);
    float *fs = reinterpret_cast<float *>(stage + 2 * T::TILE);
    if (wave == 0)
        dma_row_f32<MODE>(fs, lse2g + static_cast<long long>(x.bh) * L, i0, L, lane);
    else if (wave == 1)
        dma_row_f32<MODE>(fs + T::BM, ndeltag + static_cast<long long>(x.bh) * L, i0, L, lane);
}


}  // namespace dd
