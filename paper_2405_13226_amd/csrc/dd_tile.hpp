// dd_tile.hpp -- LDS tiles for gfx950: row-major bf16 tiles filled by direct
// global->LDS DMA, read either row-wise (ds_read_b128) or transposed
// (ds_read_b64_tr_b16), both free of LDS bank conflicts.
//
// A tile holds ROWS token rows x D head dims of one (b, h) slice, row pitch D
// elements (no padding).  Rows are split into 16-byte chunks (8 elements);
// logical chunk x of row r is stored at chunk x ^ swz(r).  The swizzle makes
// two access patterns hit 64 distinct 4-byte banks per 256-byte LDS cycle:
//   * row reads: 16 lanes read the same logical chunk of 16 consecutive rows;
//   * transposed reads: 16 lanes read a 4-row x 16-column block (each lane 8
//     bytes), two such blocks side by side per 32 lanes.
// gfx950's LDS has 64 banks of 4 bytes.
//
// ds_read_b64_tr_b16 (measured on gfx950): within each group of 16 lanes,
// source lane 4*e + c supplies 4 elements of row e, columns 4c..4c+3 of a
// 4 x 16 block; destination lane n receives column n: rows 0..3.
#pragma once

#include "dd_device.hpp"

namespace dd {

template <int D>
__device__ __forceinline__ int swz(int r)
{
    if constexpr (D == 128)
        return ((r & 3) << 2) | ((r >> 2) & 3);
    else
        return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Element offset of (row r, column col) with col a multiple of 4.
template <int D>
__device__ __forceinline__ int tile_off(int r, int col)
{
    return r * D + (((col >> 3) ^ swz<D>(r)) << 3) + (col & 7);
}

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ lds_void *to_lds(const void *p)
{
    return (lds_void *)(p);
}

// Direct global->LDS loads through inline assembly (DmaPlan modes kDmaAsm
// and kDmaAsmCast, dma_row_f32).  Lane i's SIZE bytes from `g` land at LDS
// byte address m0 + i * SIZE, with m0 the wave-uniform `lds_base`.  Issued
// through the builtin instead, the loads make the compiler wait for all of
// them (vmcnt(0)) before every later ds_read_b64_tr_b16 of the wave, whatever
// LDS it reads: in a double-buffered tile loop that is a wait for the next
// tile's prefetch in the middle of the current tile.  The compiler does not
// know what the assembly writes, so every tile is read only after the
// wait_vmem() and the workgroup barrier that follow its loads (as all callers
// do).  Register allocation differs between the forms, so each kernel takes
// the one measured faster.
enum DmaMode {
    kDmaBuiltin = 0,  // __builtin_amdgcn_global_load_lds
    kDmaAsm = 1,      // assembly; the wave's LDS slots from scalar arithmetic
    kDmaAsmCast = 2,  // assembly; each slot's LDS address through an address-space cast
};

// LDS byte address of a generic pointer into LDS, wave-uniform: the low 32
// bits of a flat LDS address are its LDS address (the shared aperture is
// 4 GiB aligned), so no null check of an address-space cast is needed.
__device__ __forceinline__ uint32_t lds_base_sgpr(const void *p)
{
    return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}

// The same through an address-space cast (generic null maps to -1).
__device__ __forceinline__ uint32_t lds_base_cast(const void *p)
{
    return __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>(to_lds(p))));
}

__device__ __forceinline__ void dma_b128(const void *g, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(lds_base), "v"(g)
                 : "m0", "memory");
}

// The same with a wave-uniform base address and a 32-bit per-lane byte
// offset (no 64-bit address arithmetic per load).  The offsets of a tile
// fit: at most 256 rows of H * D < 2^23 elements of 2 bytes.
__device__ __forceinline__ void dma_b128_off(const void *base, uint32_t off, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(lds_base), "v"(off), "s"(base)
                 : "m0", "memory");
}

__device__ __forceinline__ void dma_b32(const void *g, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off"
                 :
                 : "s"(lds_base), "v"(g)
                 : "m0", "memory");
}

// Direct-to-LDS loads of one tile.  Every wave of the workgroup (NW waves)
// takes a share of the 64-slot (1 KiB) load instructions; slot q of the tile
// holds row q / (D/8), stored chunk q % (D/8).  The byte offsets of a wave's
// slots relative to the tile's first global row are computed once; a tile
// that runs past row L-1 takes a slow path that clamps rows to L-1 (their
// values are finite and the mask removes them).  Completion is tracked by
// vmcnt.
template <int D, int ROWS, int NW, int MODE = kDmaBuiltin>
struct DmaPlan {
    static constexpr int CPR = D / 8;               // chunks per row
    static constexpr int INSTRS = ROWS * CPR / 64;  // wave instructions per tile
    static constexpr int PER = INSTRS / NW;         // per wave
    static_assert(INSTRS % NW == 0, "tile loads must divide over the waves");
    uint32_t off[PER];

    __device__ __forceinline__ void init(long long rs, int wave, int lane)
    {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int q = (wave + NW * k) * 64 + lane;
            const int r = q / CPR, x = (q % CPR) ^ swz<D>(r);
            off[k] = static_cast<uint32_t>((r * rs + x * 8) * 2);
        }
    }

    __device__ __forceinline__ void issue(uint16_t *lds_tile, const uint16_t *__restrict__ g,
                                          long long rs, int row0, int L, int wave, int lane) const
    {
        // kDmaAsm: the wave's first 1 KiB slot of the tile, in SGPRs.
        const uint32_t lslot =
            MODE == kDmaAsm ? lds_base_sgpr(lds_tile) +
                                  1024u * static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(wave))
                            : 0u;
        auto slot = [&](int k) __attribute__((always_inline)) -> uint32_t {
            return MODE == kDmaAsm ? lslot + 1024u * NW * k
                                   : lds_base_cast(lds_tile + (wave + NW * k) * 512);
        };
        if (row0 + ROWS <= L) {
            const char *gb = reinterpret_cast<const char *>(g + row0 * rs);
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                if constexpr (MODE != kDmaBuiltin)
                    dma_b128_off(gb, off[k], slot(k));
                else
                    __builtin_amdgcn_global_load_lds(gb + off[k],
                                                     to_lds(lds_tile + (wave + NW * k) * 512), 16,
                                                     0, 0);
            }
        } else {
            // kDmaAsm: offsets from row min(row0, L-1), never negative and
            // below ROWS rows (a 64-bit address per lane would hold VGPRs).
            const int rb = min(row0, L - 1);
            const char *gr = reinterpret_cast<const char *>(g + rb * rs);
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                const int q = (wave + NW * k) * 64 + lane;
                const int r = q / CPR, x = (q % CPR) ^ swz<D>(r);
                const int row = min(row0 + r, L - 1);
                if constexpr (MODE == kDmaAsm)
                    dma_b128_off(gr, static_cast<uint32_t>(((row - rb) * rs + x * 8) * 2), slot(k));
                else if constexpr (MODE == kDmaAsmCast)
                    dma_b128(g + row * rs + x * 8, slot(k));
                else
                    __builtin_amdgcn_global_load_lds(g + row * rs + x * 8,
                                                     to_lds(lds_tile + (wave + NW * k) * 512), 16,
                                                     0, 0);
            }
        }
    }
};

// Direct-to-LDS load of ROWS consecutive fp32 values (ROWS == 64: one wave
// instruction of 4-byte slots), rows clamped to L-1.
template <int MODE>
__device__ __forceinline__ void dma_row_f32(float *lds, const float *__restrict__ g, int row0,
                                            int L, int lane)
{
    const int row = min(row0 + lane, L - 1);
    if constexpr (MODE == kDmaAsm)
        dma_b32(g + row, lds_base_sgpr(lds));
    else if constexpr (MODE == kDmaAsmCast)
        dma_b32(g + row, lds_base_cast(lds));
    else
        __builtin_amdgcn_global_load_lds(g + row, to_lds(lds), 4, 0, 0);
}

// Wait for this wave's outstanding vector-memory operations (incl. LDS DMA).
__device__ __forceinline__ void wait_vmem()
{
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0), expcnt/lgkmcnt unconstrained
}

__device__ __forceinline__ bf16x8 lds_row8(const uint16_t *p)
{
    return as_bf16x8(*reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ bf16x4 lds_tr4(const uint16_t *p)
{
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4 *)(p));
    return __builtin_bit_cast(bf16x4, v);
}

}  // namespace dd
