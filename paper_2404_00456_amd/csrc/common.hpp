// Shared device helpers and internal launch declarations of libquarot.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

namespace quarot {

// Output variants of the rotate kernels.
enum Epilogue : int {
    EPI_F16 = 0,  // store RN16(y)
    EPI_SYM = 1,  // per-row symmetric int4 codes + fp16 scale
    EPI_KV = 2,   // per-group asymmetric uint4 codes + fp16 scale, zero
    EPI_SYM8 = 3, // per-row symmetric codes in [-qmax-1, qmax], one byte each
    EPI_F32 = 4,  // store y in binary32 (input of the weights' clip search)
    EPI_E3M2 = 5, // EPI_SYM's codes as e3m2 numbers, tiled layout (see e3m2_head)
};

// Load stages of the rotate kernels.
enum Prologue : int {
    PRO_PLAIN = 0,   // x is the row
    PRO_SWIGLU = 1,  // the row is RN16(silu(x) * x2) (gate x, up x2)
};

// ---- int4 codes as e3m2 numbers (the operand format of the fp6 GEMM) ----
//
// These encoders are also built for the host (a CPU test runs them over all
// inputs against the format's definition), so the one device builtin they
// use, v_perm_b32, has a host stand-in written from the instruction's
// definition: the 8-byte pool {s0 (bytes 4-7), s1 (bytes 0-3)}, selector
// byte 0-7 picks a pool byte, 8-11 replicates a sign bit, 12 gives 0x00
// and larger values 0xFF.
__host__ __device__ __forceinline__ uint32_t perm_b32(uint32_t s0, uint32_t s1, uint32_t sel)
{
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_perm(s0, s1, sel);
#else
    const uint64_t pool = ((uint64_t)s0 << 32) | s1;
    uint32_t d = 0;
    for (int i = 0; i < 4; ++i) {
        const uint32_t c = (sel >> (8 * i)) & 0xFFu;
        uint32_t byte;
        if (c < 8)
            byte = (uint32_t)(pool >> (8 * c)) & 0xFFu;
        else if (c < 12)
            byte = ((pool >> (c == 8 ? 15 : c == 9 ? 31 : c == 10 ? 47 : 63)) & 1u) ? 0xFFu : 0u;
        else
            byte = c == 12 ? 0x00u : 0xFFu;
        d |= byte << (8 * i);
    }
    return d;
#endif
}
//
// e3m2: sign, 3 exponent bits (bias 3), 2 mantissa bits; every integer in
// -8..8 is exact.  For such an integer q, the binary32 encoding b of q has
// exponent field e and top mantissa bits m with 4 e + m = 4 (E + 124) + M
// for q's e3m2 exponent field E and mantissa M (|q| >= 1), so the code is
// (b >> 21 & 0x3FF) - 496, clamped at 0 for q = 0, plus the sign at bit 5.
__host__ __device__ __forceinline__ uint32_t e3m2_of_bits(uint32_t b)
{
    const int mag = (int)((b >> 21) & 0x3FFu) - 4 * 124;
    return (uint32_t)(mag > 0 ? mag : 0) | ((b >> 26) & 0x20u);
}

__device__ __forceinline__ uint32_t e3m2_of_int(int q)
{
    return e3m2_of_bits(__float_as_uint((float)q));
}

// 8 int4 codes (a dword of two's complement nibbles, low nibble first) ->
// their e3m2 codes as 48 bits (code e at bit 6e): lo = bits 0-31, hi =
// bits 32-47.  Byte lookups: v_perm_b32 picks, per byte, one of 8 table
// bytes (the codes of q = 0..7, or of q = -8..-1), and the nibble's sign bit
// chooses between the two lookups.
__host__ __device__ __forceinline__ uint32_t e3m2_lut4(uint32_t x)  // 4 nibbles, one per byte
{
    const uint32_t sel = x & 0x07070707u;
    const uint32_t pos = perm_b32(0x17161514u, 0x12100C00u, sel);  // q = 0..7
    const uint32_t neg = perm_b32(0x2C303234u, 0x35363738u, sel);  // q = -8..-1
    const uint32_t m = x & 0x08080808u;
    const uint32_t mask = (m << 3) - (m >> 3);  // 0x3F in the bytes whose q < 0
    return (neg & mask) | (pos & ~mask);
}

__host__ __device__ __forceinline__ void e3m2_of_nibbles8(uint32_t w, uint32_t &lo, uint32_t &hi)
{
    const uint32_t a = e3m2_lut4(w & 0x0F0F0F0Fu);         // codes 0, 2, 4, 6
    const uint32_t b = e3m2_lut4((w >> 4) & 0x0F0F0F0Fu);  // codes 1, 3, 5, 7
    // 12-bit pairs (c_2i | c_2i+1 << 6): pairs 0, 2 and pairs 1, 3 at bits 0, 16
    const uint32_t p02 = (a & 0x00FF00FFu) | ((b & 0x00FF00FFu) << 6);
    const uint32_t p13 = ((a >> 8) & 0x00FF00FFu) | (((b >> 8) & 0x00FF00FFu) << 6);
    lo = (p02 & 0xFFFu) | ((p13 & 0xFFFu) << 12) | (p02 << 8 & 0xFF000000u);
    hi = ((p02 >> 24) & 0xFu) | ((p13 >> 16) << 4);
}

// 32 int4 codes (four nibble dwords) -> the 192-bit unit sum_e e3m2(q_e) << 6e
// as six dwords.
__host__ __device__ __forceinline__ void e3m2_unit(const uint32_t (&w)[4], uint32_t (&o)[6])
{
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        e3m2_of_nibbles8(w[k], lo[k], hi[k]);
    o[0] = lo[0];
    o[1] = hi[0] | (lo[1] << 16);
    o[2] = (lo[1] >> 16) | (hi[1] << 16);
    o[3] = lo[2];
    o[4] = hi[2] | (lo[3] << 16);
    o[5] = (lo[3] >> 16) | (hi[3] << 16);
}

// ---- exact integer digits of fp16 values (large-m rotation m-factor) ----

// The exact integer N = t * 2^24 of an fp16 value t (bits h) as signed
// base-64 digits, N = sum_k d_k 64^k, returned as a 64-bit word whose byte k
// is d_k (int8).  t = +-mant 2^(sh - 24) with an 11-bit mant and sh in
// [0, 29]; with q = sh / 6 and r = sh - 6 q, mant << r (below 2^17) has
// three base-64 digits, which land at positions q .. q + 2 (q <= 4), all
// of them negated for negative t.  Every digit lies in [-63, 63].
__host__ __device__ __forceinline__ uint64_t f16_planes(uint32_t h)
{
    const uint32_t e = (h >> 10) & 31u;
    const uint32_t mant = (h & 1023u) | (e ? 1024u : 0u);
    const uint32_t sh = e ? e - 1u : 0u;
    const uint32_t q = (sh * 43u) >> 8;  // sh / 6 for sh < 30
    const uint32_t mp = mant << (sh - 6u * q);
    uint32_t d = (mp & 63u) | ((mp << 2) & 0x3F00u) | ((mp << 4) & 0x1F0000u);
    // bytes below 0x80 negated in place: 0x80 - d borrows from no other byte
    if (h & 0x8000u)
        d = (0x80808080u - d) ^ 0x80808080u;
    return (uint64_t)d << (8u * q);
}

// The digit planes of four fp16 values (raw bits in r.x, r.y, low half
// first): w[k] holds digit k of the four values in its bytes 0..3.
__host__ __device__ __forceinline__ void f16x4_planes(uint2 r, uint32_t w[7])
{
    const uint64_t p0 = f16_planes(r.x & 0xFFFFu), p1 = f16_planes(r.x >> 16);
    const uint64_t p2 = f16_planes(r.y & 0xFFFFu), p3 = f16_planes(r.y >> 16);
    const uint32_t l0 = (uint32_t)p0, l1 = (uint32_t)p1, l2 = (uint32_t)p2, l3 = (uint32_t)p3;
    const uint32_t h0 = (uint32_t)(p0 >> 32), h1 = (uint32_t)(p1 >> 32);
    const uint32_t h2 = (uint32_t)(p2 >> 32), h3 = (uint32_t)(p3 >> 32);
    // perm_b32(s0, s1, sel): selector byte 0-3 picks s1's bytes, 4-7 s0's
    // pairs: {digit j of v0, of v1, digit j+1 of v0, of v1}
    const uint32_t a01 = perm_b32(l1, l0, 0x05010400u);
    const uint32_t b01 = perm_b32(l1, l0, 0x07030602u);
    const uint32_t c01 = perm_b32(h1, h0, 0x05010400u);
    const uint32_t d01 = perm_b32(h1, h0, 0x0C0C0602u);
    const uint32_t a23 = perm_b32(l3, l2, 0x05010400u);
    const uint32_t b23 = perm_b32(l3, l2, 0x07030602u);
    const uint32_t c23 = perm_b32(h3, h2, 0x05010400u);
    const uint32_t d23 = perm_b32(h3, h2, 0x0C0C0602u);
    w[0] = perm_b32(a23, a01, 0x05040100u);
    w[1] = perm_b32(a23, a01, 0x07060302u);
    w[2] = perm_b32(b23, b01, 0x05040100u);
    w[3] = perm_b32(b23, b01, 0x07060302u);
    w[4] = perm_b32(c23, c01, 0x05040100u);
    w[5] = perm_b32(c23, c01, 0x07060302u);
    w[6] = perm_b32(d23, d01, 0x05040100u);
}

// Tiled e3m2 layout of a [rows, K] code matrix: K/128 blocks of rows * 96
// bytes.  Unit u (k = 128 b + 32 u .. + 31) of row r: dwords 0-3 (head) at
// e3m2_head, dwords 4-5 (tail) at e3m2_tail.  The row-dependent slot
// swizzles make the GEMM's LDS reads of 16 rows hit distinct banks.
__host__ __device__ __forceinline__ int64_t e3m2_head(int64_t rows, int64_t r, int b, int u)
{
    return (int64_t)b * rows * 96 + r * 64 + 16 * (u ^ (int)((r >> 1) & 3));
}

__host__ __device__ __forceinline__ int64_t e3m2_tail(int64_t rows, int64_t r, int b, int u)
{
    return (int64_t)b * rows * 96 + rows * 64 + r * 32 + 8 * (u ^ (int)((r >> 2) & 3));
}

struct RotArgs {
    const uint16_t *x;   // fp16 [rows, n]
    const uint16_t *x2;  // PRO_SWIGLU: the up-projection, fp16 [rows, n]
    void *out;           // EPI_F16: fp16 [rows, n]; else uint8 codes [rows, n/2]
    uint16_t *scale;     // EPI_SYM: [rows]; EPI_KV: [rows, n/group]
    uint16_t *zero;      // EPI_KV: [rows, n/group]
    int64_t rows;
    int n;
    int group;           // EPI_KV group size
    int s0;              // first butterfly bit (0; log2(head_dim) across heads)
    float c;             // RN32(1/sqrt(n)), or RN32(1/sqrt(heads)) across heads
    float clip;
    int64_t ostride;     // EPI_KV: output row of input row r is r * ostride + ooff
    int64_t ooff;
    int qmax;            // EPI_SYM8: 2^(bits-1) - 1 (127 or 31)
};

struct KvAttnArgs {
    const uint16_t *q;  // [nq, D] rotated queries
    const uint8_t *kc;  // [nkv, s_max, D/2] codes
    const uint16_t *ks, *kz;  // [nkv, s_max, D/G]
    const uint8_t *vc;
    const uint16_t *vs, *vz;
    uint16_t *out;      // [nq, D]
    float *part;        // [nq, splits, D + 2] partial (max, sum, o) when splits > 1
    int64_t nq;
    int64_t s_max;
    int rep;            // query rows per cache row
    int seq_len;
    int D, G;
    int splits, chunk;  // sequence split: tokens [s * chunk, (s + 1) * chunk)
    float sm_scale;
};

struct SearchArgs {
    const void *y;       // binary32 rows (rotated) or fp16 rows [rows, n]
    void *q;             // codes: packed nibbles (4 bits) or one byte each
    uint16_t *scale;     // [rows]
    float *clip;         // [rows] chosen clip
    int64_t rows;
    int n;
    int ncand;           // candidates c_j = RN32((100 - j) / 100), j < ncand
};
hipError_t launch_quant_search(const SearchArgs &a, int bits, bool f32_in, hipStream_t s);

// Sequence splits of the decode attention for nq query rows (the workspace
// holds nq * splits * (D + 2) floats when splits > 1).
int kv_attn_splits(int64_t nq, int64_t seq_len);
hipError_t launch_kv_attention(const KvAttnArgs &a, hipStream_t s);

struct GemmArgs {
    const uint8_t *xq;
    const uint16_t *sx;
    const uint8_t *wq;
    const uint16_t *sw;
    uint16_t *y;
    int32_t *acc;  // may be null
    int M, N, K;
};

struct KvDeqArgs {
    const uint8_t *q;
    const uint16_t *scale;
    const uint16_t *zero;
    uint16_t *out;
    int64_t rows;
    int n;
    int group;
    float c;
};

// Launchers (return hipSuccess or the launch error).  `rotate` selects the
// rotation; sizes have been validated by the caller.
hipError_t launch_rotate(const RotArgs &a, int epi, bool rotate, int k, int m, hipStream_t s,
                         int pro = PRO_PLAIN);
// bits = 4: packed int4 codes [rows, K/2]; bits = 8: one int8 code per byte.
// bits: 4 (int4 codes), 8 (one code per byte) or 6 (int4 codes in the e3m2
// layout written by launch_pack_e3m2; K a multiple of 128).
hipError_t launch_gemm(const GemmArgs &a, hipStream_t s, int bits = 4);
// int4 codes [rows, k/2] -> e3m2 layout [rows, k/128 * 96]; k % 128 == 0.
hipError_t launch_pack_e3m2(const uint8_t *q4, uint8_t *q6, int64_t rows, int k, hipStream_t s);
// Group-wise W4A4, groups of `group` (64, 128, 256) along K, K a multiple of
// max(group, 128); a.sx [K/group, M], a.sw [K/group, N].
hipError_t launch_gemm_grouped(const GemmArgs &a, int group, hipStream_t s);
hipError_t launch_gemm_grouped_e3m2(const GemmArgs &a, int group, hipStream_t s);
// Group-wise symmetric int4 of binary32 (f32_in) or fp16 rows: codes
// [rows, n/2], scales group-major [n/group, rows].
hipError_t launch_quant_grouped(const void *y, bool f32_in, uint8_t *q, uint16_t *scale,
                                int64_t rows, int n, int group, float clip, hipStream_t s);
hipError_t launch_kv_dequant(const KvDeqArgs &a, bool inverse_rotate, hipStream_t s);
hipError_t launch_swiglu(const uint16_t *g, const uint16_t *u, uint16_t *h, int64_t count,
                         hipStream_t s);

// Device address of the fixed scratch array (QUAROT_SCRATCH_BYTES) on the
// current device; looked up on the first call per device, then cached.
hipError_t scratch_buffer(void **ptr);

// Is (k, m) covered by a compiled rotate kernel for this epilogue?
bool rotate_supported(int epi, bool rotate, int k, int m, int n, int pro = PRO_PLAIN);

// ---------------------------------------------------------------- device --

__device__ __forceinline__ float h2f(uint16_t h)
{
    return __half2float(__ushort_as_half(h));
}

// RN16 of a rounded binary32 value.  The empty asm pins f to a VGPR first:
// without it the backend folds "fp32 multiply (or add), then convert" into
// one v_fma_mix*_f16, which rounds once to fp16 instead of RN16(RN32(.)).
__device__ __forceinline__ uint16_t f2h(float f)
{
    __asm__ volatile("" : "+v"(f));
    return __half_as_ushort(__float2half_rn(f));
}

// Value of lane (lane ^ (1 << J)), J = 0..3, by DPP: quad_perm for bits 0
// and 1; for bits 2 and 3 a mirror within 8 (lane ^ 7) or 16 (lane ^ 15)
// lanes composed with a second DPP.
template <int J>
__device__ __forceinline__ float lane_xor_dpp(float v)
{
    static_assert(J >= 0 && J <= 3, "bits 0..3");
    const int vi = __float_as_int(v);
    int p;
    if constexpr (J == 0) {
        p = __builtin_amdgcn_update_dpp(vi, vi, 0xB1, 0xF, 0xF, false);  // quad_perm 1,0,3,2
    } else if constexpr (J == 1) {
        p = __builtin_amdgcn_update_dpp(vi, vi, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
    } else if constexpr (J == 2) {
        const int t = __builtin_amdgcn_update_dpp(vi, vi, 0x141, 0xF, 0xF, false);  // lane ^ 7
        p = __builtin_amdgcn_update_dpp(t, t, 0x1B, 0xF, 0xF, false);  // then ^ 3
    } else {
        const int t = __builtin_amdgcn_update_dpp(vi, vi, 0x140, 0xF, 0xF, false);  // lane ^ 15
        p = __builtin_amdgcn_update_dpp(t, t, 0x141, 0xF, 0xF, false);  // then ^ 7
    }
    return __int_as_float(p);
}

// The pair across lane bit J (4 or 5) by v_permlane{16,32}_swap: .x holds
// the value of the lane with bit J clear, .y that of the lane with it set.
template <int J>
__device__ __forceinline__ float2 lane_pair_swap(float v)
{
    static_assert(J == 4 || J == 5, "bits 4, 5");
    const unsigned u = __float_as_uint(v);
    if constexpr (J == 4) {
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
}

// Compile-time loop helper: f(std::integral_constant<int, J>) for J < N.
template <int N, int J = 0, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (J < N) {
        f(std::integral_constant<int, J>());
        static_for<N, J + 1>(f);
    }
}

// ---- butterflies across lanes --------------------------------------------
//
// A row segment of L = 2^LOGL lanes holds positions 0..L-1 (the lane bits of
// the element index).  Lane l holds position pos(l) = l ^ 3*b2(l) ^ 4*b3(l)
// (b2, b3 the bits 2 and 3 of l).  With this placement the DPP patterns that
// exist on gfx950 pair the right positions: quad_perm swaps position bits 0
// and 1, row_half_mirror (l -> l^7) flips position bit 2 and row_mirror
// (l -> l^15) flips position bit 3.
__device__ __forceinline__ int lane_pos(int lane)
{
    return lane ^ (((lane >> 2) & 1) * 3) ^ (((lane >> 3) & 1) * 4);
}

// +1 where position bit J is clear, -1 where it is set.
__device__ __forceinline__ float pos_sign(int pos, int J)
{
    return ((pos >> J) & 1) ? -1.0f : 1.0f;
}

// Butterfly across position bit J < 4 as one v_fmac_f32_dpp per register:
// v <- partner * s + v with s = pos_sign(pos, J).  The lane with the bit
// clear gets u_lo + u_hi; the lane with it set gets u_hi - u_lo, the
// negative of the Walsh-Hadamard output.  Each is one rounding of an exact
// sum, and RN(-x) = -RN(x), so the lanes carry their outputs up to a known
// sign: after the DPP stages a lane holds sigma * u with
// sigma = (-1)^popcount(pos & dpp_bits), and partners in later stages share
// sigma.  The kernels fold sigma into the final scale multiply.
//
// The compiler does not fuse a DPP move into v_fmac, hence inline asm.  A
// DPP read needs two wait states after a VALU write of its source, which
// the compiler cannot see through asm: each block starts with s_nop 1, and
// within a block every instruction reads a register that no earlier one in
// the block writes.
#define QUAROT_DPP_FMAC4(CTL)                                                                \
    asm volatile("s_nop 1\n\t"                                                               \
                 "v_fmac_f32_dpp %0, %0, %4 " CTL " row_mask:0xf bank_mask:0xf\n\t"        \
                 "v_fmac_f32_dpp %1, %1, %4 " CTL " row_mask:0xf bank_mask:0xf\n\t"        \
                 "v_fmac_f32_dpp %2, %2, %4 " CTL " row_mask:0xf bank_mask:0xf\n\t"        \
                 "v_fmac_f32_dpp %3, %3, %4 " CTL " row_mask:0xf bank_mask:0xf"            \
                 : "+v"(a), "+v"(b), "+v"(c), "+v"(d)                                        \
                 : "v"(s))

template <int J>
__device__ __forceinline__ void dpp_fmac4(float &a, float &b, float &c, float &d, float s)
{
    static_assert(J >= 0 && J <= 3, "DPP butterflies cover position bits 0..3");
    if constexpr (J == 0)
        QUAROT_DPP_FMAC4("quad_perm:[1,0,3,2]");
    else if constexpr (J == 1)
        QUAROT_DPP_FMAC4("quad_perm:[2,3,0,1]");
    else if constexpr (J == 2)
        QUAROT_DPP_FMAC4("row_half_mirror");
    else
        QUAROT_DPP_FMAC4("row_mirror");
}
#undef QUAROT_DPP_FMAC4

// Four lane-pair maxima (or minima) across position bit J = 0 or 1, each
// one DPP-sourced v_max_f32 / v_min_f32 (the compiler's fmaxf of a DPP move
// adds a canonicalizing max of its own); same hazard rule as above.
#define QUAROT_DPP_MINMAX4(OP, CTL)                                                        \
    asm volatile("s_nop 1\n\t"                                                             \
                 OP "_dpp %0, %0, %0 " CTL " row_mask:0xf bank_mask:0xf\n\t"               \
                 OP "_dpp %1, %1, %1 " CTL " row_mask:0xf bank_mask:0xf\n\t"               \
                 OP "_dpp %2, %2, %2 " CTL " row_mask:0xf bank_mask:0xf\n\t"               \
                 OP "_dpp %3, %3, %3 " CTL " row_mask:0xf bank_mask:0xf"                     \
                 : "+v"(a), "+v"(b), "+v"(c), "+v"(d))

template <int J, bool MAX>
__device__ __forceinline__ void dpp_minmax4(float &a, float &b, float &c, float &d)
{
    static_assert(J == 0 || J == 1, "quad permutations only");
    if constexpr (MAX && J == 0)
        QUAROT_DPP_MINMAX4("v_max_f32", "quad_perm:[1,0,3,2]");
    else if constexpr (MAX)
        QUAROT_DPP_MINMAX4("v_max_f32", "quad_perm:[2,3,0,1]");
    else if constexpr (J == 0)
        QUAROT_DPP_MINMAX4("v_min_f32", "quad_perm:[1,0,3,2]");
    else
        QUAROT_DPP_MINMAX4("v_min_f32", "quad_perm:[2,3,0,1]");
}
#undef QUAROT_DPP_MINMAX4

// The lane-pair maximum of mx and minimum of mn across position bit J = 0
// or 1, one DPP-sourced instruction each (same hazard rule as above).
template <int J>
__device__ __forceinline__ void dpp_maxmin(float &mx, float &mn)
{
    static_assert(J == 0 || J == 1, "quad permutations only");
    if constexpr (J == 0)
        asm volatile("s_nop 1\n\t"
                     "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
                     "v_min_f32_dpp %1, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf"
                     : "+v"(mx), "+v"(mn));
    else
        asm volatile("s_nop 1\n\t"
                     "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
                     "v_min_f32_dpp %1, %1, %1 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf"
                     : "+v"(mx), "+v"(mn));
}

// One Walsh-Hadamard stage across position bit J on R registers (R a
// multiple of 4), s = pos_sign(pos, J).  J < 4: DPP as above (flips the
// sign of the lanes with the bit set).  J = 4, 5 (lane ^ 16 by ds_swizzle,
// lane ^ 32 by ds_bpermute, both through the LDS crossbar, no LDS memory):
// v <- fma(v, s, partner), which is u_lo + u_hi or u_lo - u_hi exactly
// rounded, with no sign change.
template <int J, int R>
__device__ __forceinline__ void lane_stage(float *v, float s, int lane)
{
    static_assert(R % 4 == 0, "register count");
    if constexpr (J <= 3) {
#pragma unroll
        for (int i = 0; i < R; i += 4)
            dpp_fmac4<J>(v[i], v[i + 1], v[i + 2], v[i + 3], s);
    } else if constexpr (J == 4) {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const float p = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v[i]), 0x401F));
            v[i] = __builtin_fmaf(v[i], s, p);
        }
    } else {
        static_assert(J == 5, "lane bits 0..5");
        const int addr = (lane ^ 32) << 2;
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const float p = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(v[i])));
            v[i] = __builtin_fmaf(v[i], s, p);
        }
    }
}

// All lane stages J < LOGL (in increasing J, the canonical order) on R
// registers, skipping J < j0 (j0 uniform across the wave); returns sigma,
// the sign the lane's values now carry.
template <int LOGL, int R>
__device__ __forceinline__ float lane_stages(float *v, int lane, int pos, int j0 = 0)
{
    static_for<LOGL>([&](auto J) {
        if (J >= j0)
            lane_stage<J, R>(v, pos_sign(pos, J), lane);
    });
    constexpr int dpp_bits = (1 << (LOGL < 4 ? LOGL : 4)) - 1;
    const int done = j0 <= 0 ? dpp_bits : j0 >= 4 ? 0 : (dpp_bits & ~((1 << j0) - 1));
    return (__builtin_popcount(pos & done) & 1) ? -1.0f : 1.0f;
}

template <int J>
__device__ __forceinline__ float lane_max(float v)
{
    if constexpr (J <= 3)
        return fmaxf(v, lane_xor_dpp<J>(v));
    else {
        const float2 p = lane_pair_swap<J>(v);
        return fmaxf(p.x, p.y);
    }
}

template <int J>
__device__ __forceinline__ float lane_min(float v)
{
    if constexpr (J <= 3)
        return fminf(v, lane_xor_dpp<J>(v));
    else {
        const float2 p = lane_pair_swap<J>(v);
        return fminf(p.x, p.y);
    }
}


}  // namespace quarot
