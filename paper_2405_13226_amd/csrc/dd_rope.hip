// dd_rope.hip -- rotary position embedding of one bf16 [B, L, H, D] tensor
// (dd_rope): Y = R X, or R^T X.  One thread per 8 consecutive head dims of a
// (token, head) row (a grid-stride loop past 2^28 of them): a 16-byte load,
// four pair rotations in fp32, a 16-byte store.  The kernel is HBM-bound; X == Y is safe (each thread reads its own
// 16 bytes before writing them).
#include "dd_device.hpp"
#include "dd_rope.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_prof.hpp"
#include "dd_attn.h"

#include <algorithm>
#include <cmath>

namespace dd {

template <int D, bool INV>
__global__ void __launch_bounds__(256)
rope_kernel(const uint16_t *__restrict__ X, uint16_t *__restrict__ Y, int B, int L, int H,
            RopeEpi rt, const int32_t *__restrict__ cu, int n_docs, int doc)
{
    constexpr int CG = D / 8;  // 8-dim chunks per row
    const long long total = static_cast<long long>(B) * L * H * CG;
    const long long stride = static_cast<long long>(gridDim.x) * 256;
    for (long long gid = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x; gid < total;
         gid += stride) {
        const int cg = static_cast<int>(gid % CG);
        const long long tok = gid / CG / H;
        const int i = static_cast<int>(tok % L);
        const int b = static_cast<int>(tok / L);
        int pos = i;
        if (doc && cu != nullptr) {
            int ds, de;
            doc_span(b, L, i, cu, n_docs, ds, de);
            pos = i - ds;
        }
        const bf16x8 x = as_bf16x8(*reinterpret_cast<const u32x4 *>(X + gid * 8));
        bf16x8 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float s, c;
            rope_sincos(rope_theta_j(rt, cg * 4 + e), pos, s, c);
            float x0 = static_cast<float>(x[2 * e]), x1 = static_cast<float>(x[2 * e + 1]);
            rope_pair<INV>(x0, x1, s, c);
            y[2 * e] = static_cast<__bf16>(x0);
            y[2 * e + 1] = static_cast<__bf16>(x1);
        }
        *reinterpret_cast<u32x4 *>(Y + gid * 8) = __builtin_bit_cast(u32x4, y);
    }
}

#define DD_ROPE_ARGS                                                                             \
    const uint16_t *__restrict__, uint16_t *__restrict__, int, int, int, RopeEpi,               \
        const int32_t *__restrict__, int, int
template __global__ void rope_kernel<64, false>(DD_ROPE_ARGS);
template __global__ void rope_kernel<64, true>(DD_ROPE_ARGS);
template __global__ void rope_kernel<128, false>(DD_ROPE_ARGS);
template __global__ void rope_kernel<128, true>(DD_ROPE_ARGS);
#undef DD_ROPE_ARGS

RopeEpi rope_epi(double base, int D)
{
    const double rho = std::pow(base, -2.0 / D);
    return RopeEpi{1.0, rho, rho * rho, rho * rho * rho, std::pow(rho, 4.0), std::pow(rho, 16.0)};
}

template <int D, bool INV>
static int launch_rope_d(const RopeArgs &a)
{
    // One thread per 8 dims; larger tensors loop (grid-stride), so the
    // dispatch stays far below 2^32 work-items.
    constexpr long long kMaxRopeBlocks = 1LL << 20;
    const long long threads = static_cast<long long>(a.B) * a.L * a.H * (D / 8);
    const unsigned blocks =
        static_cast<unsigned>(std::min((threads + 255) / 256, kMaxRopeBlocks));
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    ProfScope prof(K_ROPE, st);
    const hipError_t e = launch_kernel(rope_kernel<D, INV>, dim3(blocks), dim3(256), st, a.X, a.Y,
                                       a.B, a.L, a.H, rope_epi(a.base, D), a.cu, a.n_docs,
                                       a.doc ? 1 : 0);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

int launch_rope(const RopeArgs &a)
{
    if (a.D == 64)
        return a.inverse ? launch_rope_d<64, true>(a) : launch_rope_d<64, false>(a);
    return a.inverse ? launch_rope_d<128, true>(a) : launch_rope_d<128, false>(a);
}

}  // namespace dd
