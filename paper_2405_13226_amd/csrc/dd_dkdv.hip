// dd_dkdv.hip -- key-resident dK, dV of the attention backward for D = 128.
//
// This kernel is its own translation unit so that it can be built with its
// own machine-instruction scheduling strategy: scheduling for instruction-
// level parallelism measures ~6% faster on it at long sequences, while the
// same strategy slows the other backward and forward kernels.
#include "dd_bwd.hpp"
#include "dd_launch.hpp"
#include "dd_tile.hpp"

#include <algorithm>
#include <atomic>

namespace dd {

template <int D>
struct KvTile {
    static constexpr int BN = 128;            // keys per workgroup
    static constexpr int BM = 64;             // queries per tile
    static constexpr int NW = 8;              // waves: 4 key groups x 2 roles
    static constexpr int TILE = BM * D;       // elements of a Q or dO tile
    // Q tile, dO tile, then lse2[BM] and -delta[BM] as floats.
    static constexpr int STAGE = 2 * TILE + 2 * BM * 2;
    // P hand-off between the two waves of a key group: per group, 32 fp32
    // per lane (two 32-query blocks x 16 C-layout registers), 8 KiB.
    static constexpr int PBUF_FLOATS = 4 * 64 * 32;
};

// Instruction classes of __builtin_amdgcn_sched_group_barrier, and how many
// products' operands are read ahead of the matrix pipe.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr int kAhead = 4;

// Key-resident dK/dV.  The 32 keys of a group are shared by two waves on the
// same SIMD (wave w and w + 4):
//   role A (waves 0-3): K in registers; S = Q K^T, P = exp2(S*c - lse2)
//                       (masked), P handed to role B through LDS,
//                       dV^T += dO^T P;
//   role B (waves 4-7): V in registers; dP - delta = dO V^T accumulated
//                       onto -delta, dS = P (dP - delta),
//                       dK^T += Q^T dS.
// Each wave holds one accumulator set, so two waves fit per SIMD and one
// wave's softmax arithmetic overlaps the other's matrix products.
//
// PERSIST = false: one work item per workgroup (grid = all items).
// PERSIST = true: a workgroup walks its work items (item_bid) back to
// back.  During the last query tile of an item it already loads the next
// item's first Q/dO tile into the free LDS stage, and after that tile's
// mid-tile barrier (when K or V in registers is no longer needed) the next
// item's K or V rows, so the next item starts without an exposed memory
// latency.
template <int D, bool PERSIST>
__global__ void __launch_bounds__(512, 1)
dkdv_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
            const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
            const float *__restrict__ lse2g, const float *__restrict__ ndeltag,
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
    const long long rs = static_cast<long long>(H) * D;
    const int n_items = nkb * B * H;
    const int G = static_cast<int>(gridDim.x);

    int k_item = 0;
    int bid = item_bid(0, static_cast<int>(blockIdx.x), G, n_items);
    if (bid < 0)
        return;
    KvItem it = kv_item<D, T>(bid, nkb, B, L, H, causal, cu, n_docs), nit = it;

    // Per-lane state of the current item.
    int my_k, qlo_k, qhi_k, lo_w, hi_w, lo_all, hi_all;
    bool k_ok, wave_on, wave_full_keys;
    auto setup = [&](const KvItem &x) __attribute__((always_inline)) {
        const int k0w = x.kvb * T::BN + grp * 32;
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

    // Role A keeps K rows, role B keeps V rows of this lane's key
    // (B operands: column = key).
    bf16x8 kv[KK];
    // A key past L reads row L-1 instead (no branch around the loads, so
    // they stay in flight until needed): its probabilities are masked to
    // exactly 0 by a select, and its dK/dV column is never stored.
    auto load_kv = [&](const KvItem &x) __attribute__((always_inline)) {
        const int key = min(x.kvb * T::BN + grp * 32 + l32, L - 1);
        const uint16_t *src = (role_a ? K : V) + x.base + key * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            kv[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(src + kk * 16));
    };

    // Per-lane LDS offsets: row reads (row l32 of a 32-query block, chunk
    // 2*kk + g) and transposed reads (rows 8*hh + 4*g + e of a 16-query step,
    // columns db*32 + 16*(G&1) + 4*c), shared by the Q and dO tiles.
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
    // This lane's slot of the P hand-off buffer: [grp][reg/4][lane][4].
    float *pslot = pbuf + grp * 64 * 32 + lane * 4;

    f32x16 acc[DB];  // dV^T (role A) or dK^T (role B)

    // Tile loads through assembly in the one-block form; the persistent
    // form measured faster with the builtin at L = 512 and 1024.
    DmaPlan<D, T::BM, T::NW, PERSIST ? kDmaBuiltin : kDmaAsm> plan;
    plan.init(rs, wave, lane);

    // Transposed A operand (rows of the 16-query step of (qb, t2)) times a
    // bf16 B operand, accumulated into acc.
    // Issue order (enforced below): the operands of the first kAhead
    // products, then one product per pair of reads, so that LDS latency
    // overlaps the matrix pipe; fenced off from the surrounding code.
    auto tr_products = [&](const uint16_t *tile, const bf16x8 (&bop)[2][2]) {
        __builtin_amdgcn_sched_barrier(0);
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
        constexpr int N = 4 * DB;  // products
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * kAhead, 0);
#pragma unroll
        for (int i = 0; i < N - kAhead; ++i) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, kAhead, 0);
        __builtin_amdgcn_sched_barrier(0);
    };

    // Row-wise products X K^T (role A, X = Q) or X V^T (role B, X = dO).
    // The two 32-query blocks' chains alternate; same issue order as above,
    // one read per product.
    // c[qb] += (tile rows qb*32..qb*32+31) . (this wave's register rows)^T.
    auto row_products = [&](const uint16_t *tile, f32x16 (&c)[2]) {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
                c[qb] = mfma32(lds_row8(tile + qb * 32 * D + roff[kk]), kv[kk], c[qb]);
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, kAhead, 0);
#pragma unroll
        for (int i = 0; i < 2 * KK - kAhead; ++i) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, kAhead, 0);
    };

    // Phase 1 of a tile.  Role A: S, P (masked when MASKED), P to LDS and
    // to bf16.  Role B: dP.  Phase 2 (after a barrier): role A dV, role B
    // dS and dK.  With `reload`, every wave loads K or V of the next item
    // between the phases, where its rows in registers are no longer needed.
    auto body = [&](int i0, auto bufc, auto maskc, bool active, bool reload) {
        constexpr int BUF = decltype(bufc)::value;
        constexpr bool MASKED = decltype(maskc)::value != 0;
        const uint16_t *qs = lds + BUF * T::STAGE;
        const uint16_t *dos = qs + T::TILE;
        const float *lse_s = reinterpret_cast<const float *>(qs + 2 * T::TILE);
        const float *ndl_s = lse_s + T::BM;
        f32x16 c[2];
        bf16x8 bop[2][2];
        if (role_a) {
            if (active) {
                // S first: raised issue priority lets role A's products take
                // the shared matrix pipe ahead of role B's dP, so that dP runs
                // during A's softmax instead of before it (measured: 3-5%
                // faster in the persistent form, 1% slower in the other).
                if constexpr (PERSIST) {
                    __builtin_amdgcn_sched_barrier(0);
                    __builtin_amdgcn_s_setprio(3);
                    __builtin_amdgcn_sched_barrier(0);
                }
                c[0] = f32x16{};
                c[1] = f32x16{};
                row_products(qs, c);
                if constexpr (PERSIST) {
                    __builtin_amdgcn_sched_barrier(0);
                    __builtin_amdgcn_s_setprio(0);
                    __builtin_amdgcn_sched_barrier(0);
                }
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
        } else {
            if (active) {
                // dP accumulates onto -delta of its rows (register 4*rg + e
                // holds query qb*32 + 8*rg + 4*g + e): the products give
                // dP - delta directly.
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg) {
                        const f32x4 nz = *reinterpret_cast<const f32x4 *>(
                            ndl_s + qb * 32 + 8 * rg + 4 * g);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            c[qb][4 * rg + e] = nz[e];
                    }
                __builtin_amdgcn_sched_barrier(0);
                row_products(dos, c);
            }
        }
        __syncthreads();  // P visible to role B
        if (reload)
            load_kv(nit);
        if (role_a) {
            if (active)
                tr_products(dos, bop);  // dV^T += dO^T P
        } else {
            if (active) {
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg) {
                        const f32x4 pv = *reinterpret_cast<const f32x4 *>(pslot + (qb * 4 + rg) * 256);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            c[qb][4 * rg + e] = pv[e] * c[qb][4 * rg + e];
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
    auto compute = [&](int t, auto bufc, bool reload) {
        const int i0 = t * T::BM;
        const bool active = wave_on && i0 <= hi_w && i0 + T::BM - 1 >= lo_w;
        if (wave_full_keys && i0 >= lo_all && i0 + T::BM - 1 <= hi_all)
            body(i0, bufc, IC<0>{}, active, reload);
        else
            body(i0, bufc, IC<1>{}, active, reload);
    };

    // dK (scaled, and with respect to the unrotated keys under RoPE) and dV
    // of the current item.
    auto store = [&]() __attribute__((always_inline)) {
        if (k_ok && !role_a && rope != 0) {
            // Keeps the frequency arithmetic here: hoisted out of the item
            // loop it would hold ~24 registers across every tile.
            int gl = g;
            RopeEpi r = rt;
            asm volatile("" : "+v"(gl), "+s"(r.p0), "+s"(r.p1), "+s"(r.p2), "+s"(r.p3),
                         "+s"(r.r4), "+s"(r.r16));
            rope_unrotate_acc<DB>(acc, r, rope_position(it.b, L, my_k, cu, n_docs, rope), gl);
        }
        // Every lane takes part in the store's lane exchange.
        const float osc = role_a ? 1.0f : scale;
        uint16_t *dst = (role_a ? dV : dK) + it.base + static_cast<long long>(k_ok ? my_k : 0) * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db)
            store_block_bf16(dst + db * 32, acc[db], osc, g, k_ok);
    };

    setup(it);
    load_kv(it);
#pragma unroll
    for (int db = 0; db < DB; ++db)
        acc[db] = f32x16{};
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
        compute(t, bufc, more);
        wait_vmem();
        __syncthreads();
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
#pragma unroll
        for (int db = 0; db < DB; ++db)
            acc[db] = f32x16{};
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

#define DD_KV_ARGS                                                                               \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        const uint16_t *__restrict__, const float *__restrict__, const float *__restrict__,      \
        uint16_t *__restrict__, uint16_t *__restrict__, int, int, int, int,                      \
        const int32_t *__restrict__, int, float, float, int, RopeEpi, int
template __global__ void dkdv_kernel<128, false>(DD_KV_ARGS);
template __global__ void dkdv_kernel<128, true>(DD_KV_ARGS);
#undef DD_KV_ARGS

int device_cu_count()
{
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 0;
    if (dev < kMaxDevices) {
        const int v = cache[dev].load(std::memory_order_relaxed);
        if (v > 0)
            return v;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    if (dev < kMaxDevices)
        cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

hipError_t launch_dkdv_paired(const BwdArgs &a, const BwdScalars &s)
{
    using T = KvTile<128>;
    const int nkb = (a.L + T::BN - 1) / T::BN;
    const long long n_items = static_cast<long long>(nkb) * a.B * a.H;
    const long long all = (n_items + kXcds - 1) / kXcds * kXcds;
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    // Persistent for short rows, as many workgroups as are resident at once
    // (one per CU); one item per workgroup otherwise, or when that many
    // workgroups already cover every item.
    const long long pgrid =
        a.L <= kPersistMaxSpan ? persistent_grid<dkdv_kernel<128, true>>(64 * T::NW) : 0;
    const bool persist = pgrid > 0 && pgrid < all;
    return launch_kernel(persist ? dkdv_kernel<128, true> : dkdv_kernel<128, false>,
                         dim3(static_cast<unsigned>(persist ? pgrid : all)), dim3(64 * T::NW), st,
                         a.Q, a.K, a.V, a.dO, s.lse2, s.ndelta, a.dK, a.dV, a.B, a.L, a.H,
                         a.causal ? 1 : 0, a.cu, a.n_docs, s.scale_log2, s.scale, nkb, s.rt,
                         s.rope);
}

}  // namespace dd
