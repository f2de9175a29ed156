// dd_block.hip -- the elementwise and normalisation steps of one OpenLM
// transformer block around the attention: LayerNorm (forward and backward,
// with the weight and bias gradients) and the SwiGLU of the MLP.  All are
// HBM-bound passes over [rows, d] bf16 tensors with fp32 arithmetic.
//
// LayerNorm: one wave per row.  A lane holds d / 64 consecutive-in-chunks
// elements of the row (16-byte chunks at lane + 64 c), the mean and the
// biased variance are two wave reductions, and y = (x - mean) * rstd * w + b
// with rstd = 1 / sqrt(var + eps).  The backward forms, per row,
//   xhat = (x - mean) rstd,  g = dy w,
//   dx = rstd (g - mean(g) - xhat mean(g xhat))  (+ an optional residual
//   gradient added before rounding),
// and accumulates dy xhat and dy per column over the rows of a workgroup
// into an fp32 partial row of a workspace; a second kernel sums the partial
// rows into dw and db.
#include "dd_device.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_attn.h"

#include <algorithm>
#include <cmath>

namespace dd {

namespace {

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ void unpack8(const u32x4 &u, float (&f)[8])
{
    const bf16x8 b = as_bf16x8(u);
#pragma unroll
    for (int i = 0; i < 8; ++i)
        f[i] = static_cast<float>(b[i]);
}

__device__ __forceinline__ u32x4 pack8f(const float (&f)[8])
{
    bf16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        b[i] = static_cast<__bf16>(f[i]);
    return __builtin_bit_cast(u32x4, b);
}

}  // namespace

constexpr int kLnWaves = 4;       // waves (rows in flight) per workgroup
constexpr int kLnRowsPerWg = 64;  // rows per workgroup in the backward

// CH = d / 512 chunks of 8 elements per lane.
template <int CH>
__global__ void __launch_bounds__(64 * kLnWaves)
layernorm_fwd_kernel(const uint16_t *__restrict__ X, const uint16_t *__restrict__ W,
                     const uint16_t *__restrict__ Bv, uint16_t *__restrict__ Y,
                     float *__restrict__ mean_out, float *__restrict__ rstd_out, int rows, float eps)
{
    constexpr int d = CH * 512;
    const int lane = threadIdx.x & 63;
    const int row = static_cast<int>(blockIdx.x) * kLnWaves + (threadIdx.x >> 6);
    if (row >= rows)
        return;
    const uint16_t *x = X + static_cast<long long>(row) * d;
    float v[CH][8];
#pragma unroll
    for (int c = 0; c < CH; ++c)
        unpack8(*reinterpret_cast<const u32x4 *>(x + (lane + 64 * c) * 8), v[c]);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int i = 0; i < 8; ++i)
            s += v[c][i];
    const float mean = wave_sum(s) / d;
    float s2 = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float t = v[c][i] - mean;
            s2 += t * t;
        }
    const float rstd = 1.0f / sqrtf(wave_sum(s2) / d + eps);
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int col = (lane + 64 * c) * 8;
        float w[8], b[8], y[8];
        unpack8(*reinterpret_cast<const u32x4 *>(W + col), w);
        unpack8(*reinterpret_cast<const u32x4 *>(Bv + col), b);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            y[i] = (v[c][i] - mean) * rstd * w[i] + b[i];
        *reinterpret_cast<u32x4 *>(Y + static_cast<long long>(row) * d + col) = pack8f(y);
    }
    if (lane == 0) {
        mean_out[row] = mean;
        rstd_out[row] = rstd;
    }
}

// Backward over kLnRowsPerWg rows per workgroup (each wave takes every
// kLnWaves-th row); partial column sums of dy * xhat and dy go to
// part[blockIdx.x][0..d) and part[blockIdx.x][d..2d).
template <int CH>
__global__ void __launch_bounds__(64 * kLnWaves)
layernorm_bwd_kernel(const uint16_t *__restrict__ X, const uint16_t *__restrict__ W,
                     const float *__restrict__ mean_in, const float *__restrict__ rstd_in,
                     const uint16_t *__restrict__ dY, const uint16_t *__restrict__ dRes,
                     uint16_t *__restrict__ dX, float *__restrict__ part, int rows)
{
    constexpr int d = CH * 512;
    __shared__ float red[kLnWaves][2][64 * CH * 8];  // per-wave column partials
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    float dw[CH][8], db[CH][8], w[CH][8];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        unpack8(*reinterpret_cast<const u32x4 *>(W + (lane + 64 * c) * 8), w[c]);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            dw[c][i] = db[c][i] = 0.f;
    }
    const int row0 = static_cast<int>(blockIdx.x) * kLnRowsPerWg;
    for (int rr = wave; rr < kLnRowsPerWg; rr += kLnWaves) {
        const int row = row0 + rr;
        if (row >= rows)
            break;
        const long long base = static_cast<long long>(row) * d;
        const float mean = mean_in[row], rstd = rstd_in[row];
        float xh[CH][8], gy[CH][8];
        float sg = 0.f, sgx = 0.f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int col = (lane + 64 * c) * 8;
            float x[8], dy[8];
            unpack8(*reinterpret_cast<const u32x4 *>(X + base + col), x);
            unpack8(*reinterpret_cast<const u32x4 *>(dY + base + col), dy);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                xh[c][i] = (x[i] - mean) * rstd;
                gy[c][i] = dy[i] * w[c][i];
                sg += gy[c][i];
                sgx += gy[c][i] * xh[c][i];
                dw[c][i] += dy[i] * xh[c][i];
                db[c][i] += dy[i];
            }
        }
        const float mg = wave_sum(sg) / d, mgx = wave_sum(sgx) / d;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int col = (lane + 64 * c) * 8;
            float out[8], r[8];
            if (dRes != nullptr)
                unpack8(*reinterpret_cast<const u32x4 *>(dRes + base + col), r);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                out[i] = rstd * (gy[c][i] - mg - xh[c][i] * mgx);
                if (dRes != nullptr)
                    out[i] += r[i];
            }
            *reinterpret_cast<u32x4 *>(dX + base + col) = pack8f(out);
        }
    }
    // Column partials of the workgroup: the waves' sums through LDS.
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            red[wave][0][(lane + 64 * c) * 8 + i] = dw[c][i];
            red[wave][1][(lane + 64 * c) * 8 + i] = db[c][i];
        }
    __syncthreads();
    float *dst = part + static_cast<long long>(blockIdx.x) * 2 * d;
    for (int col = threadIdx.x; col < 2 * d; col += 64 * kLnWaves) {
        const int which = col >= d, cc = col - which * d;
        float s = 0.f;
#pragma unroll
        for (int wv = 0; wv < kLnWaves; ++wv)
            s += red[wv][which][cc];
        dst[col] = s;
    }
}

// Column sums of the nparts partial rows, in two stages so that the 16 MB
// of partials (65,536 rows, d = 2048) are read by many workgroups at once:
// stage 1, workgroup (x, y) sums the partial rows of chunk y (every
// kLnChunks-th group of rows) for columns 64 x .. +63 (one coalesced
// 256-byte row piece per wave and row, the four waves taking every fourth
// row, combined through LDS) into sums[y][..]; stage 2 adds the kLnChunks
// chunk sums of a column and rounds dw, db to bf16.
constexpr int kLnChunks = 32;

__global__ void __launch_bounds__(256)
layernorm_param_chunk_kernel(const float *__restrict__ part, int nparts, int d,
                             float *__restrict__ sums)
{
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = static_cast<int>(blockIdx.x) * 64 + lane;
    const int per = (nparts + kLnChunks - 1) / kLnChunks;
    const int p0 = static_cast<int>(blockIdx.y) * per, p1 = min(p0 + per, nparts);
    float s0 = 0.f, s1 = 0.f;
    if (col < 2 * d) {
        int p = p0 + wave;
        for (; p + 4 < p1; p += 8) {
            s0 += part[static_cast<long long>(p) * 2 * d + col];
            s1 += part[static_cast<long long>(p + 4) * 2 * d + col];
        }
        if (p < p1)
            s0 += part[static_cast<long long>(p) * 2 * d + col];
    }
    red[wave][lane] = s0 + s1;
    __syncthreads();
    if (wave == 0 && col < 2 * d)
        sums[static_cast<long long>(blockIdx.y) * 2 * d + col] =
            (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

__global__ void __launch_bounds__(256)
layernorm_param_grad_kernel(const float *__restrict__ sums, int d, uint16_t *__restrict__ dW,
                            uint16_t *__restrict__ dB)
{
    const int col = static_cast<int>(blockIdx.x) * 256 + threadIdx.x;
    if (col >= 2 * d)
        return;
    float s = 0.f;
#pragma unroll 8
    for (int c = 0; c < kLnChunks; ++c)
        s += sums[static_cast<long long>(c) * 2 * d + col];
    const __bf16 v = static_cast<__bf16>(s);
    uint16_t *dst = col < d ? dW + col : dB + (col - d);
    *dst = __builtin_bit_cast(uint16_t, v);
}

// SwiGLU: y = silu(u) * v, silu(u) = u / (1 + exp(-u)); 8 elements per
// thread, grid-stride.
__global__ void __launch_bounds__(256)
swiglu_fwd_kernel(const uint16_t *__restrict__ U, const uint16_t *__restrict__ V,
                  uint16_t *__restrict__ Y, long long n8)
{
    const long long stride = static_cast<long long>(gridDim.x) * 256;
    for (long long t = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x; t < n8; t += stride) {
        float u[8], v[8], y[8];
        unpack8(*reinterpret_cast<const u32x4 *>(U + t * 8), u);
        unpack8(*reinterpret_cast<const u32x4 *>(V + t * 8), v);
#pragma unroll
        for (int i = 0; i < 8; ++i)
            y[i] = u[i] / (1.0f + __expf(-u[i])) * v[i];
        *reinterpret_cast<u32x4 *>(Y + t * 8) = pack8f(y);
    }
}

// Its backward: du = dy v silu'(u), dv = dy silu(u), with
// silu'(u) = sigma(u) (1 + u (1 - sigma(u))).
__global__ void __launch_bounds__(256)
swiglu_bwd_kernel(const uint16_t *__restrict__ U, const uint16_t *__restrict__ V,
                  const uint16_t *__restrict__ dY, uint16_t *__restrict__ dU,
                  uint16_t *__restrict__ dV, long long n8)
{
    const long long stride = static_cast<long long>(gridDim.x) * 256;
    for (long long t = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x; t < n8; t += stride) {
        float u[8], v[8], dy[8], du[8], dv[8];
        unpack8(*reinterpret_cast<const u32x4 *>(U + t * 8), u);
        unpack8(*reinterpret_cast<const u32x4 *>(V + t * 8), v);
        unpack8(*reinterpret_cast<const u32x4 *>(dY + t * 8), dy);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float sg = 1.0f / (1.0f + __expf(-u[i]));
            du[i] = dy[i] * v[i] * sg * (1.0f + u[i] * (1.0f - sg));
            dv[i] = dy[i] * u[i] * sg;
        }
        *reinterpret_cast<u32x4 *>(dU + t * 8) = pack8f(du);
        *reinterpret_cast<u32x4 *>(dV + t * 8) = pack8f(dv);
    }
}

#define DD_LNF_ARGS                                                                              \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        uint16_t *__restrict__, float *__restrict__, float *__restrict__, int, float
#define DD_LNB_ARGS                                                                              \
    const uint16_t *__restrict__, const uint16_t *__restrict__, const float *__restrict__,      \
        const float *__restrict__, const uint16_t *__restrict__, const uint16_t *__restrict__,   \
        uint16_t *__restrict__, float *__restrict__, int
template __global__ void layernorm_fwd_kernel<1>(DD_LNF_ARGS);
template __global__ void layernorm_fwd_kernel<2>(DD_LNF_ARGS);
template __global__ void layernorm_fwd_kernel<4>(DD_LNF_ARGS);
template __global__ void layernorm_bwd_kernel<1>(DD_LNB_ARGS);
template __global__ void layernorm_bwd_kernel<2>(DD_LNB_ARGS);
template __global__ void layernorm_bwd_kernel<4>(DD_LNB_ARGS);
#undef DD_LNF_ARGS
#undef DD_LNB_ARGS

size_t layernorm_workspace_bytes(int rows, int d)
{
    // The workgroups' partial rows, then the chunk sums.
    const long long nparts = (rows + kLnRowsPerWg - 1) / kLnRowsPerWg;
    return static_cast<size_t>(nparts + kLnChunks) * 2 * d * sizeof(float);
}

int launch_layernorm_fwd(const LayerNormArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const dim3 grid(static_cast<unsigned>((a.rows + kLnWaves - 1) / kLnWaves)), block(64 * kLnWaves);
    const auto *X = static_cast<const uint16_t *>(a.X);
    const auto *W = static_cast<const uint16_t *>(a.w);
    const auto *Bv = static_cast<const uint16_t *>(a.b);
    auto *Y = static_cast<uint16_t *>(a.Y);
    hipError_t e;
    switch (a.d) {
    case 512: e = launch_kernel(layernorm_fwd_kernel<1>, grid, block, st, X, W, Bv, Y, a.mean, a.rstd, a.rows, a.eps); break;
    case 1024: e = launch_kernel(layernorm_fwd_kernel<2>, grid, block, st, X, W, Bv, Y, a.mean, a.rstd, a.rows, a.eps); break;
    default: e = launch_kernel(layernorm_fwd_kernel<4>, grid, block, st, X, W, Bv, Y, a.mean, a.rstd, a.rows, a.eps); break;
    }
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_layernorm_bwd(const LayerNormArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const int nparts = (a.rows + kLnRowsPerWg - 1) / kLnRowsPerWg;
    const dim3 grid(static_cast<unsigned>(nparts)), block(64 * kLnWaves);
    const auto *X = static_cast<const uint16_t *>(a.X);
    const auto *W = static_cast<const uint16_t *>(a.w);
    const auto *dY = static_cast<const uint16_t *>(a.dY);
    const auto *dR = static_cast<const uint16_t *>(a.dRes);
    auto *dX = static_cast<uint16_t *>(a.dX);
    auto *part = static_cast<float *>(a.workspace);
    hipError_t e;
    switch (a.d) {
    case 512: e = launch_kernel(layernorm_bwd_kernel<1>, grid, block, st, X, W, a.mean_in, a.rstd_in, dY, dR, dX, part, a.rows); break;
    case 1024: e = launch_kernel(layernorm_bwd_kernel<2>, grid, block, st, X, W, a.mean_in, a.rstd_in, dY, dR, dX, part, a.rows); break;
    default: e = launch_kernel(layernorm_bwd_kernel<4>, grid, block, st, X, W, a.mean_in, a.rstd_in, dY, dR, dX, part, a.rows); break;
    }
    if (e != hipSuccess)
        return DD_ERR_HIP;
    float *sums = part + static_cast<long long>(nparts) * 2 * a.d;
    e = launch_kernel(layernorm_param_chunk_kernel,
                      dim3(static_cast<unsigned>((2 * a.d + 63) / 64), kLnChunks), dim3(256), st,
                      static_cast<const float *>(part), nparts, a.d, sums);
    if (e != hipSuccess)
        return DD_ERR_HIP;
    e = launch_kernel(layernorm_param_grad_kernel, dim3(static_cast<unsigned>((2 * a.d + 255) / 256)),
                      dim3(256), st, static_cast<const float *>(sums), a.d,
                      static_cast<uint16_t *>(a.dw), static_cast<uint16_t *>(a.db));
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

// Y[c][r] = X[r][c] for a bf16 matrix, one 64 x 64 tile per workgroup:
// 16-byte row pieces of X into LDS (rows padded by 16 bytes), then each
// thread gathers eight elements of a tile column and writes them as a
// 16-byte piece of a Y row.
__global__ void __launch_bounds__(256)
transpose_kernel(const uint16_t *__restrict__ X, uint16_t *__restrict__ Y, int tiles_c,
                 long long ldx, long long ldy)
{
    constexpr int P = 72;  // LDS row pitch (elements)
    __shared__ __attribute__((aligned(16))) uint16_t t[64 * P];
    const int tid = threadIdx.x;
    const long long r0 = static_cast<long long>(blockIdx.x / tiles_c) * 64;
    const long long c0 = static_cast<long long>(blockIdx.x % tiles_c) * 64;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = tid + 256 * i, r = q >> 3, c = (q & 7) * 8;
        *reinterpret_cast<u32x4 *>(t + r * P + c) =
            *reinterpret_cast<const u32x4 *>(X + (r0 + r) * ldx + c0 + c);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = tid + 256 * i, j = q >> 3, k = (q & 7) * 8;  // Y row c0 + j, columns r0 + k ..
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[e] = static_cast<uint32_t>(t[(k + 2 * e) * P + j]) |
                   (static_cast<uint32_t>(t[(k + 2 * e + 1) * P + j]) << 16);
        *reinterpret_cast<u32x4 *>(Y + (c0 + j) * ldy + r0 + k) = w;
    }
}

int launch_transpose(const TransposeArgs &a)
{
    const int tiles_c = a.cols / 64;
    const long long tiles = static_cast<long long>(a.rows / 64) * tiles_c;
    const hipError_t e = launch_kernel(transpose_kernel, dim3(static_cast<unsigned>(tiles)),
                                       dim3(256), static_cast<hipStream_t>(a.stream),
                                       static_cast<const uint16_t *>(a.X),
                                       static_cast<uint16_t *>(a.Y), tiles_c, a.ldx, a.ldy);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_swiglu(const SwigluArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const long long n8 = a.n / 8;
    const unsigned blocks = static_cast<unsigned>(std::min<long long>((n8 + 255) / 256, 16384));
    hipError_t e;
    if (!a.backward)
        e = launch_kernel(swiglu_fwd_kernel, dim3(blocks), dim3(256), st,
                          static_cast<const uint16_t *>(a.U), static_cast<const uint16_t *>(a.V),
                          static_cast<uint16_t *>(a.Y), n8);
    else
        e = launch_kernel(swiglu_bwd_kernel, dim3(blocks), dim3(256), st,
                          static_cast<const uint16_t *>(a.U), static_cast<const uint16_t *>(a.V),
                          static_cast<const uint16_t *>(a.dY), static_cast<uint16_t *>(a.dU),
                          static_cast<uint16_t *>(a.dV), n8);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

}  // namespace dd
