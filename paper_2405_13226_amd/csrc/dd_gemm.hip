// dd_gemm.hip -- bf16 matrix products of the transformer block around the
// attention (the projections and the MLP of one OpenLM block) on gfx950
// matrix cores:  C[M, N] = op(A) op(B),  bf16 inputs, fp32 accumulation.
//
//   op(A) = A, stored [M][K] with row stride lda, or A^T with A stored [K][M]
//   op(B) = B, stored [K][N] with row stride ldb, or B^T with B stored [N][K]
//
// A forward projection y = x W is (A, B) = (x, W); the backward's input
// gradient dx = dy W^T is (dy, W^T) and its weight gradient dW = x^T dy is
// (x^T, dy).
//
// One workgroup (8 waves) computes a 256 x 256 tile of C; wave (wm, wn) owns
// rows 128 wm .. +127 and columns 64 wn .. +63, i.e. 4 x 2 blocks of the
// 32x32x16 bf16 product.  The K axis is walked in 64-wide steps: the A and B
// tiles of a step are four 64 x 64 sub-tiles each, in two LDS stages, one
// barrier per step.  Every sub-tile sits in LDS as the matrix stores it, in
// the attention kernels' swizzled row-major layout.  An operand stored with
// its reduction axis along the rows (A^T, B) is read with the transposing
// LDS read; one stored with it along the columns is read row-wise.  Both
// give a lane the 8 consecutive k of its row or column.  When both operands
// are read row-wise (A, B^T: the input gradients), the next step's
// sub-tiles arrive by direct global->LDS loads of whole 128-byte rows during
// the current step's products.  Otherwise they are
// loaded into registers (16 bytes per lane and sub-tile) during the products
// and written to the other stage after them: after a direct load the
// compiler waits for it before every transposing LDS read.
//
// Each product is issued as D = op(B)^T op(A)^T, so a lane's accumulator holds
// 4 consecutive columns of C in each register group: the epilogue writes 8
// bytes per lane and register group to an LDS copy of the tile, and the tile
// then goes to memory in full 16-byte rows.  With split-K (weight gradients,
// whose reduction axis is the 65,536 tokens), every split writes an fp32
// partial tile to the caller's workspace and a second kernel sums them.
#include "dd_device.hpp"
#include "dd_tile.hpp"
#include "dd_internal.h"
#include "dd_launch.hpp"
#include "dd_attn.h"

#include <algorithm>

namespace dd {

struct GemmTile {
    static constexpr int BM = 256, BN = 256, BK = 64, NW = 8;
    static constexpr int SUB = 64 * 64;        // elements of one 64 x 64 sub-tile
    static constexpr int HALF = 4 * SUB;       // the A (or B) tile of one K step
};

// TA: A is stored [K][M]; TB: B is stored [N][K]; PART: write an fp32
// partial tile of split blockIdx.y to P ([splits][M][N]) instead of C.
// R (optional, not with PART): a bf16 matrix with row stride ldc added to
// the rounded product before the final rounding (C may be R itself).
template <bool TA, bool TB, bool PART>
__global__ void __launch_bounds__(512, 1)
gemm_kernel(const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, uint16_t *C,
            float *__restrict__ P, const uint16_t *R, int M, int N, int K, long long lda,
            long long ldb, long long ldc, int k_len)
{
    using T = GemmTile;
    // Two K-step stages (A then B sub-tiles each), reused by the epilogue.
    __shared__ __attribute__((aligned(1024))) uint16_t lds[4 * T::HALF];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
    const int wm = wave >> 2, wn = wave & 3;
    const int tiles_n = N / T::BN;
    // Workgroups are dispatched round-robin over the 8 XCDs (block id % 8),
    // each with its own L2.  Without a K split, XCD x takes the tile rows x,
    // x + 8, ..., in bands of kGR of its rows; a band is walked in groups of
    // kGC columns, each group column by column (kGR x kGC = 32 tiles, one
    // per CU of the XCD), so the tiles that run at the same time share kGR
    // A panels and kGC B panels in one L2.
    int tm, tn;
    if (gridDim.y == 1 && (M / T::BM) % kXcds == 0) {
        constexpr int kGR = 4, kGC = 8;
        const int x = static_cast<int>(blockIdx.x) % kXcds, k = static_cast<int>(blockIdx.x) / kXcds;
        const int rows_x = (M / T::BM) / kXcds;
        const int band = k / (kGR * tiles_n), rem = k % (kGR * tiles_n);
        const int gr = min(kGR, rows_x - band * kGR);  // rows of this band
        const int grp_c = rem / (gr * kGC), w = rem % (gr * kGC);
        tm = (band * kGR + w % gr) * kXcds + x;
        tn = grp_c * kGC + w / gr;
    } else {
        tm = static_cast<int>(blockIdx.x) / tiles_n;
        tn = static_cast<int>(blockIdx.x) % tiles_n;
    }
    const int m0 = tm * T::BM, n0 = tn * T::BN;
    const int kbeg = static_cast<int>(blockIdx.y) * k_len;
    const int nkt = min(k_len, K - kbeg) / T::BK;

    // A 64 x 64 sub-tile (8 KiB) is stored as the matrix stores it, rows of
    // 128 bytes in the tile_off<64> layout: an operand whose reduction axis
    // runs along the rows (A^T, B) is read with the transposing LDS read, one
    // whose reduction axis runs along the columns (A, B^T) row-wise.  (A
    // layout of 16-column slabs for the row-wise operands, conflict-free on
    // paper, measured 0.86 LDS bank-conflict cycles per LDS instruction.)
    // Every lane loads 16 bytes of each sub-tile per K step: row q / 8,
    // chunk q % 8 (q = 64 wave + lane), so a load instruction reads eight
    // whole 128-byte row pieces.  The host guarantees that every tile lies
    // inside the matrices (M, N multiples of 256, K of 64): no load needs
    // clamping.
    const int q = wave * 64 + lane, qr = q >> 3, qc = q & 7;
    const uint16_t *pa = A + qr * lda + qc * 8 +
                         (TA ? static_cast<long long>(kbeg) * lda + m0 : static_cast<long long>(m0) * lda + kbeg);
    const uint16_t *pb = B + qr * ldb + qc * 8 +
                         (TB ? static_cast<long long>(n0) * ldb + kbeg : static_cast<long long>(kbeg) * ldb + n0);
    // LDS position of this lane's chunk.
    const int wpos = qr * 64 + 8 * (qc ^ swz<64>(qr));
    // Sub-tile s starts 64 rows (stored along the tile's rows) or 64 columns
    // further; K step kt moves 64 rows or columns.
    const long long sa = TA ? 64 : 64 * lda, sb = TB ? 64 * ldb : 64;
    const long long ka = TA ? 64 * lda : 64, kb = TB ? 64 : 64 * ldb;
    u32x4 ra[4], rb[4];
    auto load = [&](int kt) __attribute__((always_inline)) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            ra[s] = *reinterpret_cast<const u32x4 *>(pa + kt * ka + s * sa);
            rb[s] = *reinterpret_cast<const u32x4 *>(pb + kt * kb + s * sb);
        }
    };
    auto store = [&](uint16_t *stage) __attribute__((always_inline)) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            *reinterpret_cast<u32x4 *>(stage + s * T::SUB + wpos) = ra[s];
            *reinterpret_cast<u32x4 *>(stage + T::HALF + s * T::SUB + wpos) = rb[s];
        }
    };

    // Transposed reads (elements within a sub-tile, sub-step 0): rows
    // 8 g + e (and + 4), columns co + 16 (G & 1) + 4 c, for column offsets
    // co = 0 and 32.
    const int G16 = lane >> 4, e4 = (lane & 15) >> 2, c4 = lane & 3;
    auto tr_off = [&](int co, int hh) __attribute__((always_inline)) {
        return tile_off<64>(8 * g + 4 * hh + e4, co + 16 * (G16 & 1) + 4 * c4);
    };
    // Fragment i of A: rows (m) 32 i .. +31 of the wave's 128, sub-tile
    // 2 wm + i / 2; fragment j of B: columns 32 j .. +31 of the wave's 64,
    // sub-tile wn.  Transposed reads of sub-step kk: + 16 rows.  Row reads:
    // rows at tile_off<64>(row, 16 kk + 8 g); the swizzle depends on the row
    // mod 16, so rows 32 further are 32 * 64 elements further.
    constexpr bool kDirect = !TA && TB;
    int dro[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
        dro[kk] = tile_off<64>(l32, 16 * kk + 8 * g);
    auto a_frag = [&](const uint16_t *at, int i, int kk) __attribute__((always_inline)) {
        const uint16_t *sub = at + (2 * wm + (i >> 1)) * T::SUB;
        const int mo = 32 * (i & 1);
        if constexpr (!TA)
            return lds_row8(sub + mo * 64 + dro[kk]);
        else
            return join(lds_tr4(sub + kk * 1024 + tr_off(mo, 0)),
                        lds_tr4(sub + kk * 1024 + tr_off(mo, 1)));
    };
    auto b_frag = [&](const uint16_t *bt, int j, int kk) __attribute__((always_inline)) {
        const uint16_t *sub = bt + wn * T::SUB;
        const int no = 32 * j;
        if constexpr (TB)
            return lds_row8(sub + no * 64 + dro[kk]);
        else
            return join(lds_tr4(sub + kk * 1024 + tr_off(no, 0)),
                        lds_tr4(sub + kk * 1024 + tr_off(no, 1)));
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = f32x16{};

    // The 32 products of a K step, with the LDS reads issued kAhead reads
    // ahead of the matrix pipe (then the rest spread over the products) so
    // that their latency overlaps earlier products (measured 3-6% faster
    // than the compiler's order).
    auto compute = [&](const uint16_t *stage) __attribute__((always_inline)) {
        const uint16_t *at = stage, *bt = stage + T::HALF;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < T::BK / 16; ++kk) {
            bf16x8 af[4], bf[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                af[i] = a_frag(at, i, kk);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[j] = b_frag(bt, j, kk);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = mfma32(bf[j], af[i], acc[i][j]);  // rows n, columns m
        }
        // reads per K step: A 16 row reads or 32 transposed halves, B 8 row
        // reads or 16 transposed halves
        constexpr int kAhead = 8;
        constexpr int NR = (TA ? 32 : 16) + (TB ? 8 : 16);
        constexpr int NP = 32;
        constexpr int QR = (NR - kAhead) / NP, RR = (NR - kAhead) % NP;
        __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
        for (int i = 0; i < RR; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, QR + 1, 0);
        }
#pragma unroll
        for (int i = RR; i < NP; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if constexpr (QR > 0)
                __builtin_amdgcn_sched_group_barrier(0x100, QR, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    if constexpr (kDirect) {
        // Sub-tile s of A (B^T): rows 64 s .. +63 of the tile's rows (columns),
        // the step's 64 k; one 1 KiB load instruction per wave and sub-tile.
        DmaPlan<64, 64, T::NW> plan_a, plan_b;
        plan_a.init(lda, wave, lane);
        plan_b.init(ldb, wave, lane);
        const uint16_t *ga = A + static_cast<long long>(m0) * lda + kbeg;
        const uint16_t *gb = B + static_cast<long long>(n0) * ldb + kbeg;
        constexpr int kNoClamp = 0x7fffffff;  // every tile lies inside the matrices
        auto dma = [&](int kt, uint16_t *stage) __attribute__((always_inline)) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                plan_a.issue(stage + s * T::SUB, ga + kt * T::BK, lda, 64 * s, kNoClamp, wave,
                             lane);
                plan_b.issue(stage + T::HALF + s * T::SUB, gb + kt * T::BK, ldb, 64 * s,
                             kNoClamp, wave, lane);
            }
        };
        dma(0, lds);
        wait_vmem();
        __syncthreads();
        for (int kt = 0; kt < nkt; ++kt) {
            if (kt + 1 < nkt)
                dma(kt + 1, lds + ((kt + 1) & 1) * 2 * T::HALF);
            compute(lds + (kt & 1) * 2 * T::HALF);
            wait_vmem();
            __syncthreads();
        }
    } else {
        load(0);
        store(lds);
        __syncthreads();
        for (int kt = 0; kt < nkt; ++kt) {
            const bool more = kt + 1 < nkt;
            if (more)
                load(kt + 1);
            compute(lds + (kt & 1) * 2 * T::HALF);
            if (more)
                store(lds + ((kt + 1) & 1) * 2 * T::HALF);
            __syncthreads();
        }
    }

    // Accumulator (i, j), register 4 q + e: column m = 32 i + l32 of the
    // wave's rows, row n = 32 j + 8 q + 4 g + e of its columns.
    if constexpr (PART) {
        float *dst = P + static_cast<long long>(blockIdx.y) * M * N;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const long long m = m0 + 128 * wm + 32 * i + l32;
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int n = n0 + 64 * wn + 32 * j + 8 * q + 4 * g;
                    f32x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[e] = acc[i][j][4 * q + e];
                    *reinterpret_cast<f32x4 *>(dst + m * N + n) = v;
                }
        }
    } else {
        // The tile in bf16 through LDS, then to memory in 16-byte pieces of
        // rows.  Rows 0..127 (waves wm = 0) go to stage 0, rows 128..255 to
        // stage 1, each 128 x 256 elements; the 4-element group n/4 of row r
        // is stored at group (n/4) ^ (2 (r mod 16)), which keeps the two
        // groups of a 16-byte piece adjacent and spreads one write
        // instruction's 32 rows over the LDS banks.
        uint16_t *ct = lds + wm * 2 * T::HALF;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 32 * i + l32;
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int n = 64 * wn + 32 * j + 8 * q + 4 * g;
                    *reinterpret_cast<bf16x4 *>(ct + r * T::BN + 4 * ((n >> 2) ^ (2 * (r & 15)))) =
                        pack4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                              acc[i][j][4 * q + 3]);
                }
        }
        __syncthreads();
#pragma unroll 4
        for (int it = 0; it < T::BM * T::BN / 8 / (64 * T::NW); ++it) {
            const int idx = it * 64 * T::NW + tid;
            const int h = idx >> 12, r = (idx >> 5) & 127, ch = idx & 31;
            const uint16_t *src = lds + h * 2 * T::HALF + r * T::BN + 8 * (ch ^ (r & 15));
            const long long at = (m0 + 128 * h + r) * ldc + n0 + ch * 8;
            u32x4 v = *reinterpret_cast<const u32x4 *>(src);
            if (R != nullptr) {
                const bf16x8 x = as_bf16x8(v), y = as_bf16x8(*reinterpret_cast<const u32x4 *>(R + at));
                bf16x8 z;
#pragma unroll
                for (int t = 0; t < 8; ++t)
                    z[t] = static_cast<__bf16>(static_cast<float>(x[t]) + static_cast<float>(y[t]));
                v = __builtin_bit_cast(u32x4, z);
            }
            *reinterpret_cast<u32x4 *>(C + at) = v;
        }
    }
}

// C = sum over splits of P (fp32 [splits][M][N]) rounded to bf16; 8 elements
// per thread, grid-stride.
__global__ void __launch_bounds__(256)
gemm_reduce_kernel(const float *__restrict__ P, uint16_t *C, const uint16_t *R, long long MN,
                   int splits, long long ldc, int N)
{
    const long long stride = static_cast<long long>(gridDim.x) * 256;
    for (long long v = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x; v < MN / 8;
         v += stride) {
        const long long e0 = v * 8;
        f32x4 s0 = *reinterpret_cast<const f32x4 *>(P + e0);
        f32x4 s1 = *reinterpret_cast<const f32x4 *>(P + e0 + 4);
        for (int s = 1; s < splits; ++s) {
            s0 += *reinterpret_cast<const f32x4 *>(P + s * MN + e0);
            s1 += *reinterpret_cast<const f32x4 *>(P + s * MN + e0 + 4);
        }
        const long long m = e0 / N, n = e0 % N;
        if (R != nullptr) {
            const bf16x8 r = as_bf16x8(*reinterpret_cast<const u32x4 *>(R + m * ldc + n));
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                s0[t] = static_cast<float>(static_cast<__bf16>(s0[t])) + static_cast<float>(r[t]);
                s1[t] = static_cast<float>(static_cast<__bf16>(s1[t])) + static_cast<float>(r[t + 4]);
            }
        }
        *reinterpret_cast<bf16x8 *>(C + m * ldc + n) =
            join(pack4(s0[0], s0[1], s0[2], s0[3]), pack4(s1[0], s1[1], s1[2], s1[3]));
    }
}

#define DD_GEMM_ARGS                                                                             \
    const uint16_t *__restrict__, const uint16_t *__restrict__, uint16_t *, float *__restrict__, \
        const uint16_t *, int, int, int, long long, long long, long long, int
template __global__ void gemm_kernel<false, false, false>(DD_GEMM_ARGS);
template __global__ void gemm_kernel<false, true, false>(DD_GEMM_ARGS);
template __global__ void gemm_kernel<true, false, false>(DD_GEMM_ARGS);
template __global__ void gemm_kernel<true, false, true>(DD_GEMM_ARGS);
template __global__ void gemm_kernel<false, false, true>(DD_GEMM_ARGS);
template __global__ void gemm_kernel<false, true, true>(DD_GEMM_ARGS);
#undef DD_GEMM_ARGS

// Splits of the K axis: enough workgroups to cover every CU about twice
// (tiles alone leave CUs idle when M N / 256^2 is small and K is long), each
// split a multiple of 64 and at least 1024 long.
int gemm_splits(int M, int N, int K)
{
    const long long tiles = static_cast<long long>(M / GemmTile::BM) * (N / GemmTile::BN);
    const int cus = std::max(device_cu_count(), 1);
    int s = 1;
    while (tiles * s < 2LL * cus && K / (2 * s) >= 1024 && (K / (2 * s)) % GemmTile::BK == 0)
        s *= 2;
    return s;
}

size_t gemm_workspace_bytes(int M, int N, int K, int splits)
{
    return splits > 1 ? static_cast<size_t>(splits) * M * N * sizeof(float) : 0;
}

int launch_gemm(const GemmArgs &a)
{
    hipStream_t st = static_cast<hipStream_t>(a.stream);
    const int splits = a.splits;
    const int k_len = a.K / splits;
    const dim3 grid(static_cast<unsigned>((a.M / GemmTile::BM) * (a.N / GemmTile::BN)),
                    static_cast<unsigned>(splits));
    const uint16_t *A = static_cast<const uint16_t *>(a.A);
    const uint16_t *B = static_cast<const uint16_t *>(a.B);
    uint16_t *C = static_cast<uint16_t *>(a.C);
    float *P = static_cast<float *>(a.workspace);
    const uint16_t *R = static_cast<const uint16_t *>(a.R);
    hipError_t e;
    const bool part = splits > 1;
#define DD_GEMM_LAUNCH(TA, TB, PT)                                                               \
    e = launch_kernel(gemm_kernel<TA, TB, PT>, grid, dim3(512), st, A, B, C, P, R, a.M, a.N,     \
                      a.K, a.lda, a.ldb, a.ldc, k_len)
    if (!a.trans_a && !a.trans_b) {
        if (part) DD_GEMM_LAUNCH(false, false, true); else DD_GEMM_LAUNCH(false, false, false);
    } else if (!a.trans_a && a.trans_b) {
        if (part) DD_GEMM_LAUNCH(false, true, true); else DD_GEMM_LAUNCH(false, true, false);
    } else {
        if (part) DD_GEMM_LAUNCH(true, false, true); else DD_GEMM_LAUNCH(true, false, false);
    }
#undef DD_GEMM_LAUNCH
    if (e != hipSuccess || !part)
        return e == hipSuccess ? DD_OK : DD_ERR_HIP;
    const long long MN = static_cast<long long>(a.M) * a.N;
    const unsigned blocks = static_cast<unsigned>(std::min<long long>((MN / 8 + 255) / 256, 8192));
    e = launch_kernel(gemm_reduce_kernel, dim3(blocks), dim3(256), st,
                      static_cast<const float *>(P), C, R, MN, splits, a.ldc, a.N);
    return e == hipSuccess ? DD_OK : DD_ERR_HIP;
}

}  // namespace dd
