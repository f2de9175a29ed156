// dd_device.hpp -- device-side building blocks shared by the attention
// kernels for gfx950 (CDNA4): vector types, the bf16 32x32x16 matrix-core
// product, bf16 packing, document-span lookup and the tile stager that fills
// LDS with both row-major and transposed copies of a 4-row x 8-column unit.
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

// Wave-wide min / max of an int.
__device__ __forceinline__ int wave_min(int v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v = min(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ int wave_max(int v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v = max(v, __shfl_xor(v, o));
    return v;
}

// ---------------------------------------------------------------------------
// Tile staging.  A tile is ROWS consecutive token rows x D columns of one
// (b, h) slice of a [B, L, H, D] bf16 tensor.  The unit of work of a thread is
// 4 rows x 8 columns (four 16-byte global loads).  A unit can be written to
// LDS row-major (pitch RP elements, one 16-byte store per row) and/or
// transposed (column-major with pitch TP elements: column c of the unit is
// one 8-byte store of the 4 rows).  Rows at or beyond L load as zeros.
// ---------------------------------------------------------------------------
struct Unit4x8 {
    u32x4 r[4];
};

template <int D>
__device__ __forceinline__ void load_unit(Unit4x8 &u, const uint16_t *__restrict__ base,
                                          long long row_stride, int row0, int L, int unit)
{
    constexpr int CG = D / 8;  // 8-column groups per row
    const int rg = unit / CG, cg = unit % CG;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = row0 + rg * 4 + i;
        if (row < L)
            u.r[i] = *reinterpret_cast<const u32x4 *>(base + row * row_stride + cg * 8);
        else
            u.r[i] = u32x4{0u, 0u, 0u, 0u};
    }
}

template <int D, int RP>
__device__ __forceinline__ void store_unit_rows(const Unit4x8 &u, uint16_t *lds, int unit)
{
    constexpr int CG = D / 8;
    const int rg = unit / CG, cg = unit % CG;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        *reinterpret_cast<u32x4 *>(lds + (rg * 4 + i) * RP + cg * 8) = u.r[i];
}

template <int D, int TP>
__device__ __forceinline__ void store_unit_cols(const Unit4x8 &u, uint16_t *lds, int unit)
{
    constexpr int CG = D / 8;
    const int rg = unit / CG, cg = unit % CG;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int w = c >> 1;
        uint32_t lo, hi;
        if ((c & 1) == 0) {
            lo = (u.r[0][w] & 0xffffu) | (u.r[1][w] << 16);
            hi = (u.r[2][w] & 0xffffu) | (u.r[3][w] << 16);
        } else {
            lo = (u.r[0][w] >> 16) | (u.r[1][w] & 0xffff0000u);
            hi = (u.r[2][w] >> 16) | (u.r[3][w] & 0xffff0000u);
        }
        *reinterpret_cast<u32x2 *>(lds + (cg * 8 + c) * TP + rg * 4) = u32x2{lo, hi};
    }
}

}  // namespace dd
