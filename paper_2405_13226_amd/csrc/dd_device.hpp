// dd_device.hpp -- device-side building blocks shared by the attention
// kernels for gfx950 (CDNA4): vector types, the bf16 32x32x16 matrix-core
// product, bf16 packing, the mask's document spans, the XCD-aware block map
// and wave reductions.
//
// Matrix-core layout used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A (32 x 16): lane l holds row l%32, k-slots 8*(l/32) .. 8*(l/32)+7
//   B (16 x 32): lane l holds col l%32, k-slots 8*(l/32) .. 8*(l/32)+7
//   C (32 x 32): lane l holds col l%32, rows 8*(r/4) + 4*(l/32) + r%4, r=0..15
// Only the row/col placement matters for correctness: A and B are always
// filled with the same slot-to-k mapping, and a reduction is invariant under
// any common permutation of k.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ bf16x8 join(bf16x4 lo, bf16x4 hi)
{
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Eight fp32 values (f[o..o+7] of a 16-vector) rounded to bf16 (RNE).
__device__ __forceinline__ bf16x8 pack8(const f32x16 &f, int o)
{
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        r[i] = static_cast<__bf16>(f[o + i]);
    return r;
}

__device__ __forceinline__ bf16x4 pack4(float a, float b, float c, float d)
{
    bf16x4 r;
    r[0] = static_cast<__bf16>(a);
    r[1] = static_cast<__bf16>(b);
    r[2] = static_cast<__bf16>(c);
    r[3] = static_cast<__bf16>(d);
    return r;
}

// Document span of row-local position p (0 <= p < L) of row b:
// [ds, de) is the part of p's document inside the row.  Without cu_doclens
// the whole row is one document.  The result is clamped to contain p, so
// malformed offsets can never produce an empty or out-of-row span.
__device__ __forceinline__ void doc_span(int b, int L, int p, const int32_t *__restrict__ cu,
                                         int n_docs, int &ds, int &de)
{
    if (cu == nullptr) {
        ds = 0;
        de = L;
        return;
    }
    const long long row0 = static_cast<long long>(b) * L;
    const long long t = row0 + p;
    int lo = 0, hi = n_docs - 1;  // largest k in [0, n_docs) with cu[k] <= t
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (static_cast<long long>(cu[mid]) <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    long long s = cu[lo], e = cu[lo + 1];
    s = s < row0 ? row0 : s;
    e = e > row0 + L ? row0 + L : e;
    int a = static_cast<int>(s - row0), z = static_cast<int>(e - row0);
    ds = (a > p || a < 0) ? p : a;
    de = (z < p + 1 || z > L) ? p + 1 : z;
}

// Allowed key interval [lo, hi] of query p (query side of the mask).
__device__ __forceinline__ void query_keys(int b, int L, int p, bool causal,
                                           const int32_t *__restrict__ cu, int n_docs,
                                           int &lo, int &hi)
{
    int ds, de;
    doc_span(b, L, p, cu, n_docs, ds, de);
    lo = ds;
    hi = causal ? p : de - 1;
}

// Allowed query interval [lo, hi] of key p (key side of the same mask).
__device__ __forceinline__ void key_queries(int b, int L, int p, bool causal,
                                            const int32_t *__restrict__ cu, int n_docs,
                                            int &lo, int &hi)
{
    int ds, de;
    doc_span(b, L, p, cu, n_docs, ds, de);
    lo = causal ? p : ds;
    hi = de - 1;
}

// Block -> (slice, block-within-slice) map.  Workgroups are dispatched
// round-robin over the 8 XCDs of the chip (block id % 8); each XCD has its
// own L2.  When the slice count is a multiple of 8, XCD x receives slices
// x, x + 8, ..., and all blocks of one slice consecutively, so the blocks
// that re-read a slice's tiles run together on one L2.  `j` counts the
// blocks of a slice in dispatch order (callers map it heaviest-first).
constexpr int kXcds = 8;

__device__ __forceinline__ void block_slice(int bid, int nblk, int BH, int &bh, int &j)
{
    if (BH % kXcds == 0) {
        const int x = bid % kXcds, n = bid / kXcds;
        bh = (n / nblk) * kXcds + x;
        j = n % nblk;
    } else {
        bh = bid % BH;
        j = bid / BH;
    }
}

// Work item k of workgroup w among G (G a multiple of 8): the block id that
// block_slice maps to a (slice, block), or -1 past the last item.  Each
// XCD's workgroups (w % 8 = x) take the XCD's block sequence n = 0, 1, ...
// (block id 8n + x) in rounds of 2C (C = G / 8 workgroups per XCD), in
// zig-zag order: workgroup c takes positions c and 2C-1-c of every round.
// Under the causal mask a slice's blocks cost linearly less (or more) work
// in block order, so each workgroup's pair of a round sums to the same cost.
__device__ __forceinline__ int item_bid(int k, int w, int G, int n_items)
{
    const int x = w % kXcds, c = w / kXcds, C = G / kXcds;
    const int n = 2 * C * (k >> 1) + ((k & 1) ? 2 * C - 1 - c : c);
    const int bid = n * kXcds + x;
    return bid < n_items ? bid : -1;
}

// Reductions over the two halves of a wave (lanes l and l ^ 32), with
// v_permlane32_swap: called with two copies of v, it returns one copy whose
// upper half received the lower half's values and one whose lower half
// received the upper half's, i.e. {v[l % 32], v[l % 32 + 32]} in every lane l.
// A VALU exchange, no LDS round trip; max and + are symmetric, so the result
// is the same in both halves.
__device__ __forceinline__ float halves_max(float v)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float v)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Stores a 32-element block of one row held in the matrix-core C layout
// (register 4*rg + e of lane (l32, g) is element 8*rg + 4*g + e of row l32),
// scaled and rounded to bf16, as 16-byte pieces: lanes l and l + 32 swap the
// halves of each pair of 8-element groups (v_permlane32_swap), after which
// lane g holds elements 8*rg .. 8*rg + 7 for rg = g and g + 2.  A store
// instruction then writes 32 contiguous bytes per row instead of 8.  `dst`
// points at element 0 of the block in this lane's row (16-byte aligned);
// every lane of the wave takes part in the exchange, and only lanes with
// `ok` store.
__device__ __forceinline__ void store_block_bf16(uint16_t *dst, const f32x16 &acc, float scale,
                                                 int g, bool ok)
{
#pragma unroll
    for (int rp = 0; rp < 2; ++rp) {
        const int r0 = 2 * rp, r1 = 2 * rp + 1;
        const bf16x4 a = pack4(acc[4 * r0] * scale, acc[4 * r0 + 1] * scale,
                               acc[4 * r0 + 2] * scale, acc[4 * r0 + 3] * scale);
        const bf16x4 b = pack4(acc[4 * r1] * scale, acc[4 * r1 + 1] * scale,
                               acc[4 * r1 + 2] * scale, acc[4 * r1 + 3] * scale);
        const u32x2 ua = __builtin_bit_cast(u32x2, a), ub = __builtin_bit_cast(u32x2, b);
        const u32x2 give = g ? ua : ub, keep = g ? ub : ua;
        u32x2 got;
#pragma unroll
        for (int w = 0; w < 2; ++w) {
            const auto r = __builtin_amdgcn_permlane32_swap(give[w], give[w], false, false);
            got[w] = g ? r[0] : r[1];
        }
        const u32x4 piece = g ? u32x4{got[0], got[1], keep[0], keep[1]}
                              : u32x4{keep[0], keep[1], got[0], got[1]};
        if (ok)
            *reinterpret_cast<u32x4 *>(dst + 8 * (g ? r1 : r0)) = piece;
    }
}

// Wave-wide min / max of an int.  Every lane ends with the same value; the
// result is taken from lane 0 so that the compiler keeps it in a scalar
// register.
__device__ __forceinline__ int wave_min(int v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v = min(v, __shfl_xor(v, o));
    return __builtin_amdgcn_readfirstlane(v);
}
__device__ __forceinline__ int wave_max(int v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v = max(v, __shfl_xor(v, o));
    return __builtin_amdgcn_readfirstlane(v);
}

// A compile-time int as a type, to select a branch of a generic lambda.
template <int N>
struct IC {
    static constexpr int value = N;
};

}  // namespace dd
