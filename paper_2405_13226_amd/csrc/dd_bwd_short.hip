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
//
// Rows of 129..256 tokens use a persistent form (bwd_short_persist_kernel):
// one workgroup per CU walks slices.  It visits the query tiles in
// descending order, so that once a tile is done its Q and dO rows, and under
// the causal mask the K rows of the tile above it, are read no more; right
// after a tile's barrier every thread loads its share of the next slice's
// rows of that tile into registers and writes them into the freed LDS rows
// after the next tile's barrier (delta and the LSE of those rows are formed
// on the way).  A slice's inputs then arrive while the previous slice
// computes, instead of in a load phase of their own (measured at L = 256,
// B*H = 4096: 0.35 ms against 0.43 ms for one workgroup per slice).
#include "dd_bwd.hpp"
#include "dd_launch.hpp"
#include "dd_tile.hpp"

#include <climits>

namespace dd {

// Per-lane LDS offsets of the short-row kernels (D = 64): row reads (row l32 of
// a 32-row block, chunk 2*kk + g) and transposed reads (rows 8*hh + 4*g + e of
// a 16-row step, columns db*32 + 16*(G&1) + 4*c).
struct ShortOffsets {
    int roff[4], toff[2][2];
    __device__ __forceinline__ void init(int lane)
    {
        const int l32 = lane & 31, g = lane >> 5;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
            roff[kk] = tile_off<64>(l32, kk * 16 + g * 8);
        const int G16 = lane >> 4, e = (lane & 15) >> 2, c = lane & 3;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                toff[db][hh] = tile_off<64>(8 * hh + 4 * g + e, db * 32 + 16 * (G16 & 1) + 4 * c);
    }
};

// One 32-query tile (queries i0..i0+31) for this wave's 32 keys: S = Q K^T,
// P = exp2(S*scale*log2e - lse2) (masked to the lane's allowed queries
// [qlo_k, qhi_k]), dP - delta accumulated onto -delta, dS = P (dP - delta),
// dV^T += dO^T P, dK^T += Q^T dS.  Returns dS in the C layout (row = query
// 8*rg + 4*g + e, column = key).
__device__ __forceinline__ f32x16 short_tile(const uint16_t *qs, const uint16_t *dos,
                                             const float *lse_s, const float *ndl_s, int i0,
                                             const bf16x8 (&kf)[4], const bf16x8 (&vf)[4],
                                             const ShortOffsets &o, int qlo_k, int qhi_k, int g,
                                             float scale_log2, f32x16 (&dk)[2], f32x16 (&dv)[2])
{
    constexpr int D = 64;
    f32x16 s = f32x16{}, ds;
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
        const f32x4 nz = *reinterpret_cast<const f32x4 *>(ndl_s + i0 + 8 * rg + 4 * g);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            ds[4 * rg + e] = nz[e];
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const int off = i0 * D + o.roff[kk];
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
        for (int db = 0; db < 2; ++db) {
            const int ro = (i0 + 16 * t2) * D;
            const bf16x8 ado = join(lds_tr4(dos + ro + o.toff[db][0]),
                                    lds_tr4(dos + ro + o.toff[db][1]));
            const bf16x8 aq = join(lds_tr4(qs + ro + o.toff[db][0]),
                                   lds_tr4(qs + ro + o.toff[db][1]));
            dv[db] = mfma32(ado, pb, dv[db]);
            dk[db] = mfma32(aq, sb, dk[db]);
        }
    }
    return ds;
}

// Writes this wave's dS of a tile into the dS rows of its keys: columns
// 0..31 of a D-wide row for even tiles, 32..63 for odd ones.
__device__ __forceinline__ void short_put_ds(uint16_t *dss, const f32x16 &ds, int wave, int lane,
                                             int qt)
{
    const int kr = wave * 32 + (lane & 31), g = lane >> 5, half = 32 * (qt & 1);
#pragma unroll
    for (int rg = 0; rg < 4; ++rg)
        *reinterpret_cast<bf16x4 *>(dss + tile_off<64>(kr, half + 8 * rg + 4 * g)) =
            pack4(ds[4 * rg], ds[4 * rg + 1], ds[4 * rg + 2], ds[4 * rg + 3]);
}

// dQ^T of the tile's queries i0..i0+31, head dims db*32..db*32+31, = K^T dS^T
// over the keys [klo, khi] the tile's queries see (keys of other documents in
// that range have dS = 0); both operands read transposed from LDS; written
// scaled, in bf16.
__device__ __forceinline__ void short_dq(const uint16_t *ks, const uint16_t *dss,
                                         const ShortOffsets &o, int db, int qt, int klo, int khi,
                                         int L, long long rs, uint16_t *__restrict__ dQs,
                                         int lane, float scale)
{
    constexpr int D = 64;
    const int l32 = lane & 31, g = lane >> 5, i0 = qt * 32;
    // Columns 32 further on flip bit 5 of a swizzled offset (the chunk's bit
    // 2, which the swizzle of D = 64 tiles keeps), so the offsets of head
    // dims db*32.. and of the odd tiles' dS columns follow from toff[0] by
    // arithmetic (no indexing of the offset arrays by a run-time value).
    const int a0 = o.toff[0][0] ^ (32 * db), a1 = o.toff[0][1] ^ (32 * db);
    const int t0 = o.toff[0][0] ^ (32 * (qt & 1)), t1 = o.toff[0][1] ^ (32 * (qt & 1));
    f32x16 acc = f32x16{};
    for (int kb = klo / 16; kb <= khi / 16; ++kb) {
        const uint16_t *kr = ks + kb * 16 * D;
        const uint16_t *sr = dss + kb * 16 * D;
        const bf16x8 a = join(lds_tr4(kr + a0), lds_tr4(kr + a1));
        const bf16x8 bs = join(lds_tr4(sr + t0), lds_tr4(sr + t1));
        acc = mfma32(a, bs, acc);
    }
    const int q = i0 + l32;
    store_block_bf16(dQs + static_cast<long long>(min(q, L - 1)) * rs + db * 32, acc, scale, g,
                     q < L);
}

// dK (scaled) and dV of this lane's key my_k (stored only when ok: a key
// inside the row; every lane takes part in the exchange).
__device__ __forceinline__ void short_store_kv(const f32x16 (&dk)[2], const f32x16 (&dv)[2],
                                               uint16_t *__restrict__ dKs,
                                               uint16_t *__restrict__ dVs, int my_k, long long rs,
                                               int g, float scale, bool ok)
{
    const long long row = ok ? my_k : 0;
    uint16_t *dKb = dKs + row * rs;
    uint16_t *dVb = dVs + row * rs;
#pragma unroll
    for (int db = 0; db < 2; ++db) {
        store_block_bf16(dKb + db * 32, dk[db], scale, g, ok);
        store_block_bf16(dVb + db * 32, dv[db], 1.0f, g, ok);
    }
}

// ROWS (64 or 128) is the row capacity: ROWS / 32 waves of 32 keys, and LDS
// for ROWS rows (33 or 65 KiB), so that shorter rows run more workgroups per
// CU; one workgroup per (b, h) slice.
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

    // Allowed queries of this lane's key, and their union over the wave's keys.
    int qlo_k = 1, qhi_k = 0;
    if (k_ok)
        key_queries(b, L, my_k, causal, cu, n_docs, qlo_k, qhi_k);
    const int lo_w = wave_min(k_ok ? qlo_k : INT_MAX);
    const int hi_w = wave_max(k_ok ? qhi_k : -1);

    ShortOffsets o;
    o.init(lane);

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
        // dS of this wave's 32 keys; zero where the wave has none.
        f32x16 ds = f32x16{};
        if (i0 <= hi_w && i0 + 31 >= lo_w)
            ds = short_tile(qs, dos, lse_s, ndl_s, i0, kf, vf, o, qlo_k, qhi_k, g, scale_log2,
                            dk, dv);
        // The dS buffer written here was last read by the dQ pass of tile
        // qt - 2, which ended before its waves reached the previous tile's
        // barrier.
        short_put_ds(dss, ds, wave, lane, qt);
        __syncthreads();  // the tile's dS is complete

        // dQ: the last two waves have the fewest tiles under the causal
        // mask, so they take it.
        if (wave >= kSNW - DB) {
            int klo, khi, tmp;
            query_keys(b, L, i0, causal, cu, n_docs, klo, tmp);
            query_keys(b, L, min(i0 + 31, L - 1), causal, cu, n_docs, tmp, khi);
            short_dq(ks, dss, o, wave - (kSNW - DB), qt, klo, khi, L, rs, dQ + base, lane,
                     scale);
        }
    }

    short_store_kv(dk, dv, dK + base, dV + base, my_k, rs, g, scale, k_ok);
}

// -rowsum(dO * O) of one 8-element chunk pair, summed over the eight lanes
// (lane & 7 = chunk) that hold one row: the same order wherever the short
// persistent kernel forms delta.
__device__ __forceinline__ float chunk_delta(u32x4 d, u32x4 o)
{
    const bf16x8 d8 = as_bf16x8(d), o8 = as_bf16x8(o);
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        part = fmaf(static_cast<float>(d8[i]), static_cast<float>(o8[i]), part);
    part += __shfl_xor(part, 1);
    part += __shfl_xor(part, 2);
    part += __shfl_xor(part, 4);
    return -part;
}

// Persistent form for rows of 129..256 tokens (LDS for 256 rows, 130 KiB: one
// workgroup of 8 waves per CU); slices blockIdx.x, blockIdx.x + G, ...
//
// Staging: thread t < 256 stages (dO, O) chunk t % 8 of row t / 8 of a tile
// (and that row's LSE), thread t >= 256 the Q chunk of the same position,
// the K chunk of the tile above it (causal mask only) and, for tile 0, the K
// chunk of tile 0.  The swizzle of a tile row depends on its row index mod
// 16 only, so a position's LDS offset within a tile is the same in every
// tile.
__global__ void __launch_bounds__(512, 1)
bwd_short_persist_kernel(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                         const uint16_t *__restrict__ V, const uint16_t *__restrict__ O,
                         const uint16_t *__restrict__ dO, const float *__restrict__ LSE,
                         uint16_t *__restrict__ dQ, uint16_t *__restrict__ dK,
                         uint16_t *__restrict__ dV, int B, int L, int H, int causal_i,
                         const int32_t *__restrict__ cu, int n_docs, float scale_log2,
                         float scale)
{
    constexpr int ROWS = 256, D = 64, KK = D / 16, DB = D / 32;
    constexpr int kSNW = ROWS / 32, kSArr = ROWS * D;
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
    const long long rs = static_cast<long long>(H) * D;
    const int n_sl = B * H, G = static_cast<int>(gridDim.x);
    const int nqt = (L + 31) / 32;
    auto slice_base = [&](int sl) {
        return (static_cast<long long>(sl / H) * L * H + sl % H) * D;
    };

    // This thread's staging position.
    const bool pair_do = tid < 256;
    const int ur = (tid & 255) >> 3, ux = tid & 7;
    const int u_off = tile_off<D>(ur, ux * 8);  // within a tile

    ShortOffsets o;
    o.init(lane);

    int sl = static_cast<int>(blockIdx.x);
    long long base = slice_base(sl);

    // First slice: Q, dO and K by DMA, delta and lse2 through the staging
    // positions (tiles 4*(tid/256) .. +3 per thread).
    {
        DmaPlan<D, ROWS, kSNW> plan;
        plan.init(rs, wave, lane);
        plan.issue(qs, Q + base, rs, 0, L, wave, lane);
        plan.issue(dos, dO + base, rs, 0, L, wave, lane);
        plan.issue(ks, K + base, rs, 0, L, wave, lane);
        const int b0 = sl / H, h0 = sl % H;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int t = 4 * (tid >> 8) + j;
            const int row = min(32 * t + ur, L - 1);
            const long long at = base + static_cast<long long>(row) * rs + ux * 8;
            const float nd = chunk_delta(*reinterpret_cast<const u32x4 *>(dO + at),
                                         *reinterpret_cast<const u32x4 *>(O + at));
            if (ux == 0) {
                ndl_s[32 * t + ur] = nd;
                lse_s[32 * t + ur] =
                    LSE[(static_cast<long long>(b0) * L + row) * H + h0] * kLog2e;
            }
        }
    }
    bf16x8 kf[KK], vf[KK];
    auto load_v = [&](long long at_base) __attribute__((always_inline)) {
        const long long at =
            at_base + static_cast<long long>(min(wave * 32 + l32, L - 1)) * rs + g * 8;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            vf[kk] = as_bf16x8(*reinterpret_cast<const u32x4 *>(V + at + kk * 16));
    };
    // K rows of this lane's key from LDS (rows past L hold row L-1).
    auto read_k = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            kf[kk] = lds_row8(ks + wave * 32 * D + o.roff[kk]);
    };
    load_v(base);
    wait_vmem();
    __syncthreads();
    read_k();

    // Staged values of one tile position of the next slice: the (dO, O)
    // chunks and the row's LSE, or the Q chunk, the K chunk of the tile above
    // and (tile 0) the K chunk of the tile itself.
    u32x4 st0, st1, st2;
    float st_lse = 0.f;
    auto stage_load = [&](long long nbase, int nsl, int t, bool k_above, bool k_here)
        __attribute__((always_inline)) {
        const int row = min(32 * t + ur, L - 1);
        const long long at = nbase + static_cast<long long>(row) * rs + ux * 8;
        if (pair_do) {
            st0 = *reinterpret_cast<const u32x4 *>(dO + at);
            st1 = *reinterpret_cast<const u32x4 *>(O + at);
            if (ux == 0)
                st_lse = LSE[(static_cast<long long>(nsl / H) * L + row) * H + nsl % H];
        } else {
            st0 = *reinterpret_cast<const u32x4 *>(Q + at);
            if (k_above) {
                const int row1 = min(32 * (t + 1) + ur, L - 1);
                st1 = *reinterpret_cast<const u32x4 *>(K + nbase + static_cast<long long>(row1) * rs +
                                                       ux * 8);
            }
            if (k_here)
                st2 = *reinterpret_cast<const u32x4 *>(K + at);
        }
    };
    auto stage_store = [&](int t, bool k_above, bool k_here) __attribute__((always_inline)) {
        const int at = 32 * t * D + u_off;
        if (pair_do) {
            *reinterpret_cast<u32x4 *>(dos + at) = st0;
            const float nd = chunk_delta(st0, st1);
            if (ux == 0) {
                ndl_s[32 * t + ur] = nd;
                lse_s[32 * t + ur] = st_lse * kLog2e;
            }
        } else {
            *reinterpret_cast<u32x4 *>(qs + at) = st0;
            if (k_above)
                *reinterpret_cast<u32x4 *>(ks + at + 32 * D) = st1;
            if (k_here)
                *reinterpret_cast<u32x4 *>(ks + at) = st2;
        }
    };

    for (;;) {
        const int b = sl / H;
        const int nsl = sl + G;
        const bool more = nsl < n_sl;
        const long long nbase = more ? slice_base(nsl) : 0;

        const int my_k = wave * 32 + l32;
        const bool k_ok = my_k < L;
        int qlo_k = 1, qhi_k = 0;
        if (k_ok)
            key_queries(b, L, my_k, causal, cu, n_docs, qlo_k, qhi_k);
        const int lo_w = wave_min(k_ok ? qlo_k : INT_MAX);
        const int hi_w = wave_max(k_ok ? qhi_k : -1);

        f32x16 dk[DB], dv[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            dk[db] = f32x16{};
            dv[db] = f32x16{};
        }

        for (int qt = nqt - 1; qt >= 0; --qt) {
            const int i0 = qt * 32;
            f32x16 ds = f32x16{};
            if (i0 <= hi_w && i0 + 31 >= lo_w)
                ds = short_tile(qs, dos, lse_s, ndl_s, i0, kf, vf, o, qlo_k, qhi_k, g,
                                scale_log2, dk, dv);
            // The dS buffer written here was last read by the dQ pass of
            // tile qt + 2.
            short_put_ds(dss, ds, wave, lane, qt);
            __syncthreads();  // the tile's dS is complete
            // Into LDS: the next slice's rows of tile qt + 1 (its main
            // products ended before the previous barrier) and, under the
            // causal mask, K rows of tile qt + 2 (read only by dQ passes of
            // tiles >= qt + 2, which ended before the previous barrier too;
            // the dQ pass of tile qt, running alongside, reads K rows below
            // 32*(qt+1)).  Then the loads of tile qt's rows, which arrive
            // during the next tile.  Without the causal mask every dQ pass
            // reads all K rows: the next slice's K is loaded after the slice.
            if (more && qt + 1 < nqt)
                stage_store(qt + 1, causal && qt + 2 < nqt, false);
            if (more)
                stage_load(nbase, nsl, qt, causal && qt + 1 < nqt, causal && qt == 0);
            if (wave >= kSNW - DB) {
                int klo, khi, tmp;
                query_keys(b, L, i0, causal, cu, n_docs, klo, tmp);
                query_keys(b, L, min(i0 + 31, L - 1), causal, cu, n_docs, tmp, khi);
                short_dq(ks, dss, o, wave - (kSNW - DB), qt, klo, khi, L, rs, dQ + base, lane,
                         scale);
            }
        }

        short_store_kv(dk, dv, dK + base, dV + base, my_k, rs, g, scale, k_ok);
        if (!more)
            break;
        __syncthreads();  // every tile and dQ pass of this slice is done
        stage_store(0, causal && nqt > 1, causal);
        if (!causal) {
            DmaPlan<D, ROWS, kSNW> plan;
            plan.init(rs, wave, lane);
            plan.issue(ks, K + nbase, rs, 0, L, wave, lane);
        }
        load_v(nbase);
        wait_vmem();
        __syncthreads();
        read_k();
        sl = nsl;
        base = nbase;
    }
}

hipError_t launch_bwd_short(const BwdArgs &a, const BwdScalars &s)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const int n_sl = a.B * a.H;
    if (a.L > 128) {
        const long long pgrid = persistent_grid<bwd_short_persist_kernel>(512);
        if (pgrid <= 0)
            return hipErrorInvalidValue;
        const long long grid = std::min<long long>(pgrid, n_sl);
        return launch_kernel(bwd_short_persist_kernel, dim3(static_cast<unsigned>(grid)),
                             dim3(512), st, a.Q, a.K, a.V, a.O, a.dO, a.LSE, a.dQ, a.dK, a.dV,
                             a.B, a.L, a.H, a.causal ? 1 : 0, a.cu, a.n_docs, s.scale_log2,
                             s.scale);
    }
    const auto kern = a.L <= 64 ? bwd_short_kernel<64> : bwd_short_kernel<128>;
    const int rows = a.L <= 64 ? 64 : 128;
    return launch_kernel(kern, dim3(static_cast<unsigned>(n_sl)), dim3(2 * rows), st, a.Q, a.K,
                         a.V, a.O, a.dO, a.LSE, a.dQ, a.dK, a.dV, a.B, a.L, a.H,
                         a.causal ? 1 : 0, a.cu, a.n_docs, s.scale_log2, s.scale);
}

}  // namespace dd
