// dd_fwd.hip -- forward of masked causal attention (dataset decomposition
// buckets and the document-masked concat-and-chunk baseline) on gfx950.
//
// One workgroup = 4 waves = BM = 128 queries of one (b, h) slice; each wave
// owns 32 queries and keeps their Q rows in registers as matrix-core B
// operands.  The workgroup walks the key tiles (BN = 64 keys) that the mask
// allows for its queries.  K and V tiles arrive in LDS by direct
// global->LDS DMA (row-major, XOR-swizzled), double-buffered: the next tile's
// loads are in flight while the current one is consumed.
//
// Per wave and tile the product is computed transposed: S^T = K Q^T puts one
// query per lane column, so the softmax row max/sum is an in-lane reduction
// plus one exchange with lane l^32, and P^T stays in registers as the B
// operand of O^T += V^T P^T, whose A operand is read transposed from the
// row-major V tile (ds_read_b64_tr_b16).  The online softmax keeps a running max m and
// sum l in fp32 (log2 domain), rescaling the O accumulator when m grows.
// Key tiles entirely outside the mask are never visited; tiles entirely
// inside it skip the element mask (only boundary tiles evaluate it), and in
// a boundary tile a wave skips a 32-key block none of its queries sees.
#include "dd_device.hpp"
#include "dd_tile.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_prof.hpp"
#include "dd_rope.hpp"
#include "dd_attn.h"

#include <algorithm>

namespace dd {

template <int D>
struct FwdTile {
    static constexpr int BM = 128;            // queries per workgroup
    static constexpr int BN = 64;             // keys per tile
    static constexpr int TILE = BN * D;       // elements of one K or V tile
    static constexpr int STAGE = 2 * TILE;    // K then V
};

// Rescaling of the output accumulator is skipped until the running maximum
// has grown by more than this many log2 units; probabilities then stay below
// 2^8, and the final normalisation uses the same reference, so the result is
// unchanged.
constexpr float kRescaleSlack = 8.0f;

// Row lengths (tokens) up to which the forward runs persistently: 1024 at
// D = 64 (the one-block form, four waves per SIMD, is faster from 2048 on),
// 2048 at D = 128.  The test ignores document masking: documents make the
// work per query block uneven, which hardware dispatch balances and a fixed
// walk order does not.
template <int D>
constexpr long long kFwdPersistMaxSpan = D == 64 ? 1024 : 2048;

// A query-block work item of the forward: one block of FwdTile::BM queries of
// one (b, h) slice and the key tiles those queries see.
struct FwdItem {
    int b, bh, qb, t_begin, t_end;
    long long base;  // element offset of (b, row 0, h, 0)
};

template <int D>
__device__ __forceinline__ FwdItem fwd_item(int bid, int nqb, int B, int L, int H, bool causal,
                                            const int32_t *__restrict__ cu, int n_docs)
{
    using T = FwdTile<D>;
    FwdItem it;
    int jb;
    block_slice(bid, nqb, B * H, it.bh, jb);
    it.qb = nqb - 1 - jb;  // heaviest query blocks (the last) first
    it.b = it.bh / H;
    it.base = (static_cast<long long>(it.b) * L * H + it.bh % H) * D;
    // Key range: union over the block's queries (monotone in the query).
    const int qf = it.qb * T::BM, ql = min(qf + T::BM - 1, L - 1);
    int wlo, whi, tmp;
    query_keys(it.b, L, qf, causal, cu, n_docs, wlo, tmp);
    query_keys(it.b, L, ql, causal, cu, n_docs, tmp, whi);
    it.t_begin = wlo / T::BN;
    it.t_end = whi / T::BN;
    return it;
}

// PERSIST = false: one query block per workgroup.  PERSIST = true (short
// rows): a workgroup walks its query blocks in the order of item_bid; during
// a block's last key tile it DMAs the next block's first K/V tile into the
// free stage and (D = 64) the next block's Q rows into an LDS area of their
// own, read into registers after that tile (at D = 128 the Q rows are loaded
// from memory after the tile: the extra 32 KiB of LDS would cost a
// workgroup per CU).
// ROPE = true: Q holds the unrotated queries; each lane rotates its Q row
// fragments right after loading them (positions and frequencies as
// dd_rope, so the result is bit-identical to a dd_rope pass) and, when
// Qrot is not null, writes the rotated rows there for the backward.
// Waves per SIMD: four in the one-block D = 64 form (at most 128 VGPRs),
// three in the persistent one (its LDS holds three workgroups per CU), two
// at D = 128.
template <int D, bool PERSIST, bool ROPE>
__global__ void __launch_bounds__(256, D == 64 ? (PERSIST ? 3 : 4) : 2)
fwd_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
           const uint16_t *__restrict__ V, uint16_t *__restrict__ O, float *__restrict__ LSE,
           int B, int L, int H, int causal_i, const int32_t *__restrict__ cu, int n_docs,
           float scale_log2, int nqb, uint16_t *__restrict__ Qrot, RopeEpi rt, int rope)
{
    using T = FwdTile<D>;
    constexpr int KK = D / 16;  // k-steps of S^T
    constexpr int DB = D / 32;  // 32-row blocks of O^T
    // Persistent D = 64: the next item's Q rows are staged here by direct
    // loads during the current item's last tile (the register budget of
    // three waves per SIMD has no room for a second set of Q fragments).
    constexpr bool kQStage = PERSIST && D == 64;
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * T::STAGE + (kQStage ? T::BM * D : 0)];

    const bool causal = causal_i != 0;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const long long rs = static_cast<long long>(H) * D;  // token stride
    const int n_items = nqb * B * H;
    const int G = static_cast<int>(gridDim.x);

    int k_item = 0;
    const int bid = item_bid(0, static_cast<int>(blockIdx.x), G, n_items);
    if (bid < 0)
        return;
    FwdItem it = fwd_item<D>(bid, nqb, B, L, H, causal, cu, n_docs), nit = it;

    // This lane's query and its allowed keys (per item).
    int my_q, lo_q, hi_q, lo_w, hi_w, lo_all, hi_all;
    bool q_ok, wave_on, wave_full_rows;
    auto setup = [&](const FwdItem &x) __attribute__((always_inline)) {
        const int q0w = x.qb * T::BM + wave * 32;
        my_q = q0w + l32;
        q_ok = my_q < L;
        lo_q = 1;  // empty for padding rows
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

    // Q fragments (B operand: column = query, k-slots = 8 head dims).  A
    // query past L reads row L-1 instead (its scores are masked out and
    // nothing of it is stored).
    bf16x8 qf8[KK];
    // from_lds: the rows were staged in LDS (kQStage), at the K-tile layout.
    auto load_q = [&](const FwdItem &x, bool from_lds) __attribute__((always_inline)) {
        const int q_raw = x.qb * T::BM + wave * 32 + l32;
        const int q = min(q_raw, L - 1);
        const uint16_t *src = Q + x.base + q * rs + g * 8;
        if (kQStage && from_lds) {
            const uint16_t *qs = lds + 2 * T::STAGE + wave * 32 * D;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                qf8[kk] = lds_row8(qs + tile_off<D>(l32, kk * 16 + g * 8));
        } else {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
                qf8[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(src + kk * 16));
        }
        if constexpr (ROPE) {
            // Fragment kk holds dims kk*16 + 8g .. +7: pairs j = 8kk + 4g + e.
            // The opaque copies keep the frequency arithmetic here, once
            // per item, instead of hoisted across the tile loop.
            int gl = g;
            RopeEpi r = rt;
            asm volatile("" : "+v"(gl), "+s"(r.p0), "+s"(r.p1), "+s"(r.p2), "+s"(r.p3),
                         "+s"(r.r4), "+s"(r.r16));
            const int pos = rope_position(x.b, L, q, cu, n_docs, rope);
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float sn, cs;
                    rope_sincos(rope_theta_j(r, 8 * kk + 4 * gl + e), pos, sn, cs);
                    float x0 = static_cast<float>(qf8[kk][2 * e]);
                    float x1 = static_cast<float>(qf8[kk][2 * e + 1]);
                    rope_pair<false>(x0, x1, sn, cs);
                    qf8[kk][2 * e] = static_cast<__bf16>(x0);
                    qf8[kk][2 * e + 1] = static_cast<__bf16>(x1);
                }
            }
            if (Qrot != nullptr && q_raw < L) {
                uint16_t *dst = Qrot + x.base + q * rs + g * 8;
#pragma unroll
                for (int kk = 0; kk < KK; ++kk)
                    *reinterpret_cast<u32x4 *>(dst + kk * 16) = __builtin_bit_cast(u32x4, qf8[kk]);
            }
        }
    };

    // Per-lane LDS offsets (elements, relative to a tile).  K row reads: row
    // l32 of a 32-key block, chunk 2*kk + g.  V transposed reads: rows
    // 8*hh + 4*g + e of a 16-key step, columns db*32 + 16*(G&1) + 4*c.
    int koff[KK], voff[DB][2];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
        koff[kk] = tile_off<D>(l32, kk * 16 + g * 8);
    {
        const int G = lane >> 4, e = (lane & 15) >> 2, c = lane & 3;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                voff[db][hh] = tile_off<D>(8 * hh + 4 * g + e, db * 32 + 16 * (G & 1) + 4 * c);
    }

    f32x16 acc[DB];
    float m_i = -INFINITY, l_i = 0.f;

    DmaPlan<D, T::BN, 4, kDmaAsm> plan;
    plan.init(rs, wave, lane);
    auto issue = [&](const FwdItem &x, int t, uint16_t *stage) __attribute__((always_inline)) {
        plan.issue(stage, K + x.base, rs, t * T::BN, L, wave, lane);
        plan.issue(stage + T::TILE, V + x.base, rs, t * T::BN, L, wave, lane);
    };

    // One tile; MASKED selects the boundary-tile variant at compile time.
    auto body = [&](int j0, auto bufc, auto maskc) {
        constexpr int BUF = decltype(bufc)::value;
        constexpr bool MASKED = decltype(maskc)::value != 0;
        const uint16_t *kt = lds + BUF * T::STAGE;
        const uint16_t *vt = kt + T::TILE;

        // A boundary tile's 32-key block that none of the wave's queries
        // sees (scores all -inf, probabilities all 0) is skipped.
        bool on[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
            on[kb] = !MASKED || !(j0 + 32 * kb > hi_w || j0 + 32 * kb + 31 < lo_w);

        // S^T = K Q^T for two 32-key blocks.
        f32x16 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x16{};
            if (on[kb]) {
#pragma unroll
                for (int kk = 0; kk < KK; ++kk)
                    s[kb] = mfma32(lds_row8(kt + kb * 32 * D + koff[kk]), qf8[kk], s[kb]);
            }
        }

        // Boundary tiles: keys outside [lo_q, hi_q] -> -inf (branch-free).
        if constexpr (MASKED) {
            const int lo_r = lo_q - j0 - 4 * g, hi_r = hi_q - j0 - 4 * g;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int kr = kb * 32 + 8 * (r >> 2) + (r & 3);
                    const bool ok = (kr >= lo_r) & (kr <= hi_r);
                    s[kb][r] = ok ? s[kb][r] : -INFINITY;
                }
        }
        // Four independent chains (max is exact, so the order is free).
        float m4[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                m4[r & 3] = fmaxf(m4[r & 3], s[kb][r]);
        const float mx = halves_max(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3])));
        const float mc = mx * scale_log2;  // log2-domain tile maximum

        // Lazy rescale: only when some lane's maximum grew past the slack.
        if (__any(mc > m_i + kRescaleSlack)) {
            const float m_new = fmaxf(m_i, mc);
            const float alpha = fast_exp2(m_i - (m_new == -INFINITY ? 0.f : m_new));
            l_i *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db)
                acc[db] *= alpha;
            m_i = m_new;
        }
        const float neg_m = m_i == -INFINITY ? 0.f : -m_i;

        float psum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (on[kb]) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float p = fast_exp2(fmaf(s[kb][r], scale_log2, neg_m));
                    s[kb][r] = p;
                    psum += p;
                }
            }
        }
        l_i += psum;

        // O^T += V^T P^T.  B operand (kb, t2): registers 8*t2..8*t2+7 of
        // s[kb] = keys kb*32 + 16*t2 + 4g + {0..3} and the same + 8; the A
        // operand reads exactly those keys transposed from the V tile.
        bf16x8 pb[2][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
                pb[kb][t2] = pack8(s[kb], 8 * t2);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            if (!on[kb])
                continue;
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const uint16_t *vr = vt + (kb * 32 + 16 * t2) * D;
                    const bf16x8 a = join(lds_tr4(vr + voff[db][0]), lds_tr4(vr + voff[db][1]));
                    acc[db] = mfma32(a, pb[kb][t2], acc[db]);
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

    // O = acc / l and the LSE of the current item.
    auto store = [&]() __attribute__((always_inline)) {
        // Every lane takes part in the row sum's and the store's lane
        // exchanges; lanes past L store nothing.
        const float l_tot = halves_sum(l_i);
        const float inv = 1.0f / l_tot;
        uint16_t *Ob = O + it.base + static_cast<long long>(q_ok ? my_q : 0) * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db)
            store_block_bf16(Ob + db * 32, acc[db], inv, g, q_ok);
        if (q_ok && g == 0)
            LSE[(static_cast<long long>(it.b) * L + my_q) * H + it.bh % H] =
                (m_i + log2f(l_tot)) * kLn2;
    };
    auto reset = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
            acc[db] = f32x16{};
        m_i = -INFINITY;
        l_i = 0.f;
    };

    setup(it);
    load_q(it, false);
    reset();
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
                nit = fwd_item<D>(nbid, nqb, B, L, H, causal, cu, n_docs);
                issue(nit, nit.t_begin, other);
                if constexpr (kQStage) {  // two 64-row halves with the tile plan
                    plan.issue(lds + 2 * T::STAGE, Q + nit.base, rs, nit.qb * T::BM, L, wave,
                               lane);
                    plan.issue(lds + 2 * T::STAGE + T::BN * D, Q + nit.base, rs,
                               nit.qb * T::BM + T::BN, L, wave, lane);
                }
            }
        }
        compute(t, bufc);
        if (!kQStage && more)  // Q of the next item (registers free after the tile)
            load_q(nit, false);
        wait_vmem();
        __syncthreads();
        if (kQStage && more) {  // the staged rows are in LDS
            load_q(nit, true);
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
        reset();
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

// Explicit instantiations: the host-side launch stubs are emitted here
// unconditionally (clang's host pass does not always emit them for templates
// only referenced through a function pointer).
#define DD_FWD_ARGS                                                                              \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        uint16_t *__restrict__, float *__restrict__, int, int, int, int,                          \
        const int32_t *__restrict__, int, float, int, uint16_t *__restrict__, RopeEpi, int
template __global__ void fwd_kernel<64, false, false>(DD_FWD_ARGS);
template __global__ void fwd_kernel<64, true, false>(DD_FWD_ARGS);
template __global__ void fwd_kernel<128, false, false>(DD_FWD_ARGS);
template __global__ void fwd_kernel<128, true, false>(DD_FWD_ARGS);
template __global__ void fwd_kernel<64, false, true>(DD_FWD_ARGS);
template __global__ void fwd_kernel<64, true, true>(DD_FWD_ARGS);
template __global__ void fwd_kernel<128, false, true>(DD_FWD_ARGS);
template __global__ void fwd_kernel<128, true, true>(DD_FWD_ARGS);
#undef DD_FWD_ARGS

template <int D, bool ROPE>
static int launch_fwd_d(const FwdArgs &a)
{
    const int nqb = (a.L + FwdTile<D>::BM - 1) / FwdTile<D>::BM;
    const long long all = (static_cast<long long>(nqb) * a.B * a.H + kXcds - 1) / kXcds * kXcds;
    const float scale_log2 = kLog2e / sqrtf(static_cast<float>(D));
    // RoPE: 0 off, 1 row positions, 2 document-local positions.
    const int rope = ROPE ? (a.rope_doc && a.cu ? 2 : 1) : 0;
    const RopeEpi rt = ROPE ? rope_epi(a.rope_base, D) : RopeEpi{};
    // Persistent for short rows: as many workgroups as are resident at once.
    const long long pgrid =
        a.L <= kFwdPersistMaxSpan<D> ? persistent_grid<fwd_kernel<D, true, ROPE>>(256) : 0;
    const bool persist = pgrid > 0 && pgrid < all;
    ProfScope prof(K_FWD, static_cast<hipStream_t>(a.stream));
    const hipError_t e = launch_kernel(
        persist ? fwd_kernel<D, true, ROPE> : fwd_kernel<D, false, ROPE>,
        dim3(static_cast<unsigned>(persist ? pgrid : all)), dim3(256),
        static_cast<hipStream_t>(a.stream), a.Q, a.K, a.V, a.O, a.LSE, a.B, a.L, a.H,
        a.causal ? 1 : 0, a.cu, a.n_docs, scale_log2, nqb, a.Qrot, rt, rope);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_fwd(const FwdArgs &a)
{
    if (a.rope_base > 0.0)
        return a.D == 64 ? launch_fwd_d<64, true>(a) : launch_fwd_d<128, true>(a);
    return a.D == 64 ? launch_fwd_d<64, false>(a) : launch_fwd_d<128, false>(a);
}

}  // namespace dd
