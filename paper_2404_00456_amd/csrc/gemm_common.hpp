// Shared pieces of the integer GEMM kernels for gfx950: block tile and
// wave constants, the int4 -> int8 operand widening, the XCD-aware tile
// order, global -> LDS DMA and s_waitcnt encoding.
#pragma once

#include "common.hpp"

namespace quarot {
namespace gemm {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int BM = 256;   // X rows per block
constexpr int BN = 256;   // W rows per block
constexpr int BKB = 64;   // packed bytes per row per k-step
constexpr int LDSR = 80;  // LDS row pitch (bytes)
constexpr int GM = 8;     // m-tiles per group in the tile order
constexpr int STAGE = (BM + BN) * LDSR;
constexpr int LDS_BYTES = 2 * STAGE;

__device__ __forceinline__ v4i widen(uint2 d)
{
    v4i r;
    r[0] = (int)((d.x << 4) & 0xF0F0F0F0u);
    r[1] = (int)(d.x & 0xF0F0F0F0u);
    r[2] = (int)((d.y << 4) & 0xF0F0F0F0u);
    r[3] = (int)(d.y & 0xF0F0F0F0u);
    return r;
}

__device__ __forceinline__ void tile_of(int bid, int nblk, int TM, int TN, int &tm, int &tn)
{
    int t = bid;
    if ((nblk & 7) == 0)
        t = (bid & 7) * (nblk >> 3) + (bid >> 3);
    const int gsize = GM * TN;
    const int g = t / gsize;
    const int first = g * GM;
    const int gm = min(TM - first, GM);
    const int r = t - g * gsize;
    tm = first + r % gm;
    tn = r / gm;
}

constexpr int THREADS = 512;
constexpr int WN = 64;   // n per wave
constexpr int NI = WN / 16;  // n slices per wave (MFMA A operands)

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from global memory straight into LDS at
// lds_base + 16 * lane.  Issued as inline asm on purpose: for the compiler's
// own LDS-DMA builtin the waitcnt pass cannot tell the DMA target from the
// stage being read and waits for every DMA before each LDS read, which
// serializes the ring.  Here only the explicit s_waitcnt below orders it.
// M0 is declared clobbered, so the compiler keeps nothing of its own in it
// across the block; the s_nop is the wait state the ISA asks for between an
// SALU write of M0 and a VMEM instruction with LDS destination.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(g), "s"(lds_base)
                 : "memory", "m0");
}

// dma16 in the SGPR-base form: lane l reads base + voff[l] (a wave-uniform
// 64-bit base, a 32-bit per-lane offset), so the per-step address update
// is scalar work.
__device__ __forceinline__ void dma16s(uint32_t voff, const void *base, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(base), "s"(lds_base)
                 : "memory", "m0");
}

// 4 bytes per lane into LDS at lds_base + 4 * lane (same rules as dma16).
__device__ __forceinline__ void dma4(const void *g, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 :
                 : "v"(g), "s"(lds_base)
                 : "memory", "m0");
}

typedef int v8i __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) uint64_t lds_u64;
typedef float v4f __attribute__((ext_vector_type(4)));

// One e3m2 operand slice of a lane: 32 codes, six dwords (head, tail).
struct Op6 {
    uint4 h;
    uint2 t;
};

// v_mfma_f32_16x16x128_f8f6f4 with both operands e3m2 (format 3), no scale.
// Every product of two codes is an integer of magnitude <= 64 and every
// partial sum an integer below 2^24, so the binary32 accumulation is exact.
__device__ __forceinline__ v4f mfma6(const Op6 &a, const Op6 &b, v4f c)
{
    const v8i av = {(int)a.h.x, (int)a.h.y, (int)a.h.z, (int)a.h.w, (int)a.t.x, (int)a.t.y, 0, 0};
    const v8i bv = {(int)b.h.x, (int)b.h.y, (int)b.h.z, (int)b.h.w, (int)b.t.x, (int)b.t.y, 0, 0};
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 3, 3, 0, 0, 0, 0);
}

// s_waitcnt immediate: vmcnt(vm) expcnt(7) lgkmcnt(lgkm) in the gfx9 layout
constexpr int waitcnt_imm(int vm, int lgkm)
{
    return (vm & 15) | (((vm >> 4) & 3) << 14) | (7 << 4) | ((lgkm & 15) << 8);
}

}  // namespace gemm
}  // namespace quarot
