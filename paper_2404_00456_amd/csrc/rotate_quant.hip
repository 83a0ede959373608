// Online Hadamard rotation fused with quantization (§3.1, §4 Stage 1b/2b,
// §5 Setup), for gfx950.
//
// A row of width n = 2^k * m is rotated as y = x . (H_{2^k} (x) H_m) * c,
// c = RN32(1/sqrt(n)), element index i = a*m + b (m fast):
//   1. the m-factor u[a,b'] = RN32(sum_b H_m[b][b'] t[a,b]), the exact sum
//      rounded once (exact in fp64 for fp16 inputs, in any order);
//   2. the Walsh-Hadamard butterflies over a in binary32, bit 0 first, each
//      output one rounded add or subtract;
//   3. one multiply by c.
// Every kernel keeps this arithmetic exactly, whatever lane, register or
// wave holds an element, so the fp32 y (and every code derived from it) is
// reproducible bit for bit.
//
// Kernels:
//   k_rot_pow2    m = 1, n = 2^k <= 32768.  Each lane owns 16-byte chunks of
//                 8 consecutive elements: i = ((cc*W + w)*L + pos)*8 + e, so
//                 bits 0-2 live in registers, the next log2(L) bits across
//                 lanes, then across the W waves (LDS), then across chunks.
//   k_rot_smallm  m = 12, 20, 28: each lane owns whole groups of m elements;
//                 the m-factor is an fp64 sum with shared partial sums.
//   k_rot_largem  m = 108, 172: the m-factor as exact integer digit
//                 products on the int8 matrix cores, the rotated row staged
//                 in LDS.
//   k_quant_plain quantization without rotation, any n multiple of 8.
//   k_kv_dequant  4-bit KV cache back to fp16, optional inverse rotation.
// Lane butterflies use the placement and sign bookkeeping of lane_stages().
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "hadamard_factors.hpp"

namespace quarot {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v6i __attribute__((ext_vector_type(6)));

__constant__ HmMfmaB<108> c_hmb108 = HmMfmaB<108>();
__constant__ HmMfmaB<172> c_hmb172 = HmMfmaB<172>();

namespace {

constexpr int ilog2(int v)
{
    int r = 0;
    while ((1 << r) < v)
        ++r;
    return r;
}

// The quantizers divide by a stored fp16 scale sf.  RN(y / sf) is formed
// with Markstein's correction from rf = RN(1 / sf), computed once per row or
// group: q0 = RN(y rf), e = y - q0 sf (exact, one fma), q = RN(q0 + e rf).
// With a correctly rounded reciprocal this equals the IEEE quotient except
// where it underflows (|q| < 2^-100), where both give code 0; checked
// against IEEE division for every positive fp16 divisor.  A zero or
// infinite scale gives code 0 (y / inf = 0 as well).
struct Divisor {
    float s, r;
    bool ok;
};

__device__ __forceinline__ Divisor make_divisor(float sf)
{
    Divisor d;
    d.s = sf;
    d.ok = sf > 0.0f && sf < __builtin_inff();
    d.r = d.ok ? 1.0f / sf : 0.0f;
    return d;
}

__device__ __forceinline__ float quotient(float y, const Divisor &d)
{
    const float q0 = y * d.r;
    const float e = __builtin_fmaf(-q0, d.s, y);
    return __builtin_fmaf(e, d.r, q0);
}

// RN(x / 15) without a division instruction: Markstein's correction from
// RN(1/15), exact for every binary32 x (checked exhaustively on the CPU).
__device__ __forceinline__ float div15(float x)
{
    const float r = 0x1.111112p-4f;  // RN32(1/15)
    const float q0 = x * r;
    return __builtin_fmaf(__builtin_fmaf(-q0, 15.0f, x), r, q0);
}

// Rounding to an integer code without conversion instructions: for t
// clamped to the code range (|t| < 2^22), t + 1.5 * 2^23 lies in
// [2^23, 2^24), where floats are spaced by 1, so the add rounds t to the
// nearest integer, ties to even, and the low bits of the sum's encoding are
// that integer in two's complement.  Clamping before rounding equals
// rounding before clamping, as the bounds are integers.
__device__ __forceinline__ uint32_t round_bits(float t)
{
    return __float_as_uint(t + 0x1.8p23f);
}

// Symmetric int4 code (§4 Stage 2b): clamp(rint_even(RN(y / sf)), -8, 7).
__device__ __forceinline__ uint32_t sym_code(float y, const Divisor &d)
{
    const uint32_t c = round_bits(fminf(fmaxf(quotient(y, d), -8.0f), 7.0f)) & 0xFu;
    return d.ok ? c : 0u;
}

// Asymmetric uint4 code: clamp(rint_even(RN(RN(y - zf) / sf)), 0, 15), as
// the low nibble of the rounding sum's encoding (whose bits 4-21 are zero),
// for packing; the caller applies the zero-or-infinite-scale rule (code 0).
__device__ __forceinline__ uint32_t asym_code_bits(float y, const Divisor &d, float zf)
{
    return round_bits(fminf(fmaxf(quotient(y - zf, d), 0.0f), 15.0f));
}

// Symmetric code with qmax levels a side, as a byte:
// clamp(rint_even(RN(y / sf)), -qmax - 1, qmax).
__device__ __forceinline__ uint32_t sym8_code(float y, const Divisor &d, float qmaxf)
{
    const uint32_t c =
        round_bits(fminf(fmaxf(quotient(y, d), -qmaxf - 1.0f), qmaxf)) & 0xFFu;
    return d.ok ? c : 0u;
}

// The 48 code bits (lo, then the low 16 of hi) of the 8 elements i0 .. i0+7
// (i0 a multiple of 8) of row r into the tiled e3m2 layout: bytes 6p .. 6p+5
// of the 24 of unit u (i0 = 128 b + 32 u + 8 p), whose bytes 0-15 are the
// head and 16-23 the tail; each lane writes one dword and one short.
__device__ __forceinline__ void store_e3m2_48(uint8_t *q, int64_t rows, int64_t r, int64_t i0,
                                              uint32_t lo, uint32_t hi)
{
    const int p = (int)(i0 >> 3) & 3, u = (int)(i0 >> 5) & 3, b = (int)(i0 >> 7);
    const int64_t h = e3m2_head(rows, r, b, u), t = e3m2_tail(rows, r, b, u);
    const bool odd = (p & 1) != 0;
    const uint32_t dw = odd ? (lo >> 16) | (hi << 16) : lo;
    const uint16_t sh = (uint16_t)(odd ? lo : hi);
    const int64_t da = p == 0 ? h : p == 1 ? h + 8 : p == 2 ? h + 12 : t + 4;
    const int64_t sa = p == 0 ? h + 4 : p == 1 ? h + 6 : p == 2 ? t : t + 2;
    *reinterpret_cast<uint32_t *>(q + da) = dw;
    *reinterpret_cast<uint16_t *>(q + sa) = sh;
}


// The symmetric epilogues: scale divisor, row stride of the codes, and the
// codes of 8 (or 4) consecutive elements starting at element i0 of a row:
// EPI_SYM packs nibbles (4 bytes per 8), EPI_SYM8 one byte per code.
template <int EPI>
__device__ __forceinline__ float sym_divisor(const RotArgs &a)
{
    return (EPI == EPI_SYM || EPI == EPI_E3M2) ? 7.0f : (float)a.qmax;
}

template <int EPI>
__device__ __forceinline__ int64_t sym_row_bytes(int64_t n)
{
    return (EPI == EPI_SYM || EPI == EPI_E3M2) ? n / 2 : n;
}

template <int EPI>
__device__ __forceinline__ void store_codes8(uint8_t *qr, int64_t i0, const float *v,
                                             const Divisor &d, float qmaxf)
{
    if constexpr (EPI == EPI_SYM) {
        uint32_t pk = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e)
            pk |= sym_code(v[e], d) << (4 * e);
        *reinterpret_cast<uint32_t *>(qr + i0 / 2) = pk;
    } else {
        uint2 pk = make_uint2(0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            pk.x |= sym8_code(v[e], d, qmaxf) << (8 * e);
            pk.y |= sym8_code(v[4 + e], d, qmaxf) << (8 * e);
        }
        *reinterpret_cast<uint2 *>(qr + i0) = pk;
    }
}

template <int EPI>
__device__ __forceinline__ void store_codes4(uint8_t *qr, int64_t i0, const float *v,
                                             const Divisor &d, float qmaxf)
{
    if constexpr (EPI == EPI_SYM) {
        const uint32_t pk = sym_code(v[0], d) | (sym_code(v[1], d) << 4) |
                            (sym_code(v[2], d) << 8) | (sym_code(v[3], d) << 12);
        *reinterpret_cast<uint16_t *>(qr + i0 / 2) = (uint16_t)pk;
    } else {
        uint32_t pk = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            pk |= sym8_code(v[e], d, qmaxf) << (8 * e);
        *reinterpret_cast<uint32_t *>(qr + i0) = pk;
    }
}

__device__ __forceinline__ void load8(const uint16_t *p, float *v)
{
    uint4 raw = *reinterpret_cast<const uint4 *>(p);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = h2f((uint16_t)(w[i] & 0xFFFFu));
        v[2 * i + 1] = h2f((uint16_t)(w[i] >> 16));
    }
}

// load8 followed by the butterfly on element bit 0, (t_2i, t_2i+1) ->
// (RN(t_2i + t_2i+1), RN(t_2i - t_2i+1)) with t = f32(x): each output is one
// v_fma_mix_f32 on the two fp16 halves of the dword, f32(a) * (+-1) + f32(b)
// rounded once, so no conversion instruction is needed.  (Written as asm:
// the compiler turns an fma by +-1 into an add of converted values.)
__device__ __forceinline__ void load8_bit0(const uint16_t *p, float *v)
{
    uint4 raw = *reinterpret_cast<const uint4 *>(p);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float sum, dif;
        // src0 = low half (sum) / high half (dif), src1 = +-1.0 as f32,
        // src2 = high half (sum) / low half (dif)
        __asm__("v_fma_mix_f32 %0, %1, 1.0, %1 op_sel:[0,0,1] op_sel_hi:[1,0,1]"
                : "=v"(sum) : "v"(w[i]));
        __asm__("v_fma_mix_f32 %0, %1, -1.0, %1 op_sel:[1,0,0] op_sel_hi:[1,0,1]"
                : "=v"(dif) : "v"(w[i]));
        v[2 * i] = sum;
        v[2 * i + 1] = dif;
    }
}

__device__ __forceinline__ void store8(uint16_t *p, const float *v)
{
    uint4 raw;
    raw.x = (uint32_t)f2h(v[0]) | ((uint32_t)f2h(v[1]) << 16);
    raw.y = (uint32_t)f2h(v[2]) | ((uint32_t)f2h(v[3]) << 16);
    raw.z = (uint32_t)f2h(v[4]) | ((uint32_t)f2h(v[5]) << 16);
    raw.w = (uint32_t)f2h(v[6]) | ((uint32_t)f2h(v[7]) << 16);
    *reinterpret_cast<uint4 *>(p) = raw;
}

__device__ __forceinline__ void load4(const uint16_t *p, float *v)
{
    uint2 raw = *reinterpret_cast<const uint2 *>(p);
    v[0] = h2f((uint16_t)(raw.x & 0xFFFFu));
    v[1] = h2f((uint16_t)(raw.x >> 16));
    v[2] = h2f((uint16_t)(raw.y & 0xFFFFu));
    v[3] = h2f((uint16_t)(raw.y >> 16));
}

__device__ __forceinline__ void store4(uint16_t *p, const float *v)
{
    uint2 raw;
    raw.x = (uint32_t)f2h(v[0]) | ((uint32_t)f2h(v[1]) << 16);
    raw.y = (uint32_t)f2h(v[2]) | ((uint32_t)f2h(v[3]) << 16);
    *reinterpret_cast<uint2 *>(p) = raw;
}

// SiLU in binary32 by a fixed sequence of IEEE operations (Cody-Waite
// reduction of exp(-g) and a degree-7 Taylor polynomial in fma; the CPU
// reference performs the same operations):
//   x = clamp(-g, -88, 88), kf = rint_even(RN(x log2 e)),
//   r = fma(-kf, LN2_HI, fma...)  (kf LN2_HI exact: LN2_HI has 16 bits),
//   E = ldexp(p(r), kf), silu(g) = RN(g / RN(1 + E)).
__device__ __forceinline__ float silu_f32(float g)
{
    const float x = fminf(fmaxf(-g, -88.0f), 88.0f);
    const float kf = rintf(x * 0x1.715476p+0f);  // RN32(1 / ln 2)
    float r = __builtin_fmaf(-kf, 0x1.62e4p-1f, x);  // ln 2 to 16 bits
    r = __builtin_fmaf(-kf, 0x1.7f7d1cp-20f, r);     // RN32(ln 2 - that)
    float p = 0x1.a01a02p-13f;                        // RN32(1/k!), k = 7 .. 2
    p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);
    p = __builtin_fmaf(p, r, 0x1.111112p-7f);
    p = __builtin_fmaf(p, r, 0x1.555556p-5f);
    p = __builtin_fmaf(p, r, 0x1.555556p-3f);
    p = __builtin_fmaf(p, r, 0.5f);
    p = __builtin_fmaf(p, r, 1.0f);
    p = __builtin_fmaf(p, r, 1.0f);
    const float e = __builtin_ldexpf(p, (int)kf);
    return g / (1.0f + e);
}

// The down-projection input h = RN16(RN(silu(g) u)), as binary32.
__device__ __forceinline__ float swiglu1(uint16_t g, uint16_t u)
{
    return h2f(f2h(silu_f32(h2f(g)) * h2f(u)));
}

// 8 (4) consecutive elements of the row at element offset off.
template <int PRO>
__device__ __forceinline__ void load_row8(const RotArgs &a, int64_t off, float *v)
{
    if constexpr (PRO == PRO_PLAIN) {
        load8(a.x + off, v);
    } else {
        const uint4 g = *reinterpret_cast<const uint4 *>(a.x + off);
        const uint4 u = *reinterpret_cast<const uint4 *>(a.x2 + off);
        const uint32_t gw[4] = {g.x, g.y, g.z, g.w}, uw[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = swiglu1((uint16_t)(gw[i] & 0xFFFFu), (uint16_t)(uw[i] & 0xFFFFu));
            v[2 * i + 1] = swiglu1((uint16_t)(gw[i] >> 16), (uint16_t)(uw[i] >> 16));
        }
    }
}

template <int PRO>
__device__ __forceinline__ void load_row4(const RotArgs &a, int64_t off, float *v)
{
    if constexpr (PRO == PRO_PLAIN) {
        load4(a.x + off, v);
    } else {
        const uint2 g = *reinterpret_cast<const uint2 *>(a.x + off);
        const uint2 u = *reinterpret_cast<const uint2 *>(a.x2 + off);
        v[0] = swiglu1((uint16_t)(g.x & 0xFFFFu), (uint16_t)(u.x & 0xFFFFu));
        v[1] = swiglu1((uint16_t)(g.x >> 16), (uint16_t)(u.x >> 16));
        v[2] = swiglu1((uint16_t)(g.y & 0xFFFFu), (uint16_t)(u.y & 0xFFFFu));
        v[3] = swiglu1((uint16_t)(g.y >> 16), (uint16_t)(u.y >> 16));
    }
}

// 8 (4) values of y at element offset off of the output: fp16 (EPI_F16) or
// binary32 (EPI_F32).
template <int EPI>
__device__ __forceinline__ void store_y8(void *out, int64_t off, const float *v)
{
    if constexpr (EPI == EPI_F16) {
        store8(static_cast<uint16_t *>(out) + off, v);
    } else {
        float4 *p = reinterpret_cast<float4 *>(static_cast<float *>(out) + off);
        p[0] = make_float4(v[0], v[1], v[2], v[3]);
        p[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
}

template <int EPI>
__device__ __forceinline__ void store_y4(void *out, int64_t off, const float *v)
{
    if constexpr (EPI == EPI_F16)
        store4(static_cast<uint16_t *>(out) + off, v);
    else
        *reinterpret_cast<float4 *>(static_cast<float *>(out) + off) =
            make_float4(v[0], v[1], v[2], v[3]);
}

// Max over the L-lane group (xor butterfly), then over the W waves.
template <int LOGL, int W>
__device__ __forceinline__ float row_absmax(float amax, int w, float *red)
{
    static_for<LOGL>([&](auto J) { amax = lane_max<J>(amax); });
    if constexpr (W > 1) {
        if ((threadIdx.x & 63) == 0)
            red[w] = amax;
        __syncthreads();
        amax = red[0];
#pragma unroll
        for (int i = 1; i < W; ++i)
            amax = fmaxf(amax, red[i]);
    }
    return amax;
}

// ------------------------------------------------------------ m = 1 -----

// HEADS: the butterflies run over element bits >= a.s0 only (log2(head_dim):
// across heads); otherwise over all bits (s0 = 0 at compile time, so that
// no stage carries a branch).
// KVROW (EPI_KV): the quantization group is the whole row.
template <int LOGL, int W, int C, int EPI, bool ROT, int PRO = PRO_PLAIN, bool HEADS = false,
          bool KVROW = false>
__global__ __launch_bounds__(W == 1 ? 256 : 64 * W) void k_rot_pow2(RotArgs a)
{
    constexpr int L = 1 << LOGL;
    constexpr int LOGW = ilog2(W);
    constexpr int RPW = (W == 1) ? 64 / L : 1;  // rows per wave
    constexpr int RPB = (W == 1) ? 4 * RPW : 1; // rows per block
    constexpr int N = 8 * L * W * C;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // position of this lane in its row segment (see lane_pos)
    const int pos = lane_pos(lane) & (L - 1);
    int64_t row;
    int w;
    if constexpr (W == 1) {
        row = (int64_t)blockIdx.x * RPB + wave * RPW + (lane >> LOGL);
        w = 0;
        if (row >= a.rows)
            return;
    } else {
        row = blockIdx.x;
        w = wave;
    }

    // plain fp16 rows rotated from bit 0 take that butterfly in the load
    constexpr bool BIT0 = ROT && PRO == PRO_PLAIN && !HEADS;
    float v[C][8];
#pragma unroll
    for (int cc = 0; cc < C; ++cc) {
        if constexpr (BIT0)
            load8_bit0(a.x + row * N + ((cc * W + w) * L + pos) * 8, v[cc]);
        else
            load_row8<PRO>(a, row * N + ((cc * W + w) * L + pos) * 8, v[cc]);
    }

    if constexpr (ROT) {
        const int s0 = HEADS ? a.s0 : 0;
        // element bits 0..2: inside each chunk
#pragma unroll
        for (int h = BIT0 ? 2 : 1, bit = BIT0 ? 1 : 0; h < 8; h <<= 1, ++bit)
            if (bit >= s0)
#pragma unroll
                for (int cc = 0; cc < C; ++cc)
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (!(e & h)) {
                            float p = v[cc][e], q = v[cc][e + h];
                            v[cc][e] = p + q;
                            v[cc][e + h] = p - q;
                        }
        // next LOGL bits: across lanes
        const float sigma = lane_stages<LOGL, 8 * C>(&v[0][0], lane, pos, s0 - 3);
        // next LOGW bits: across waves, through LDS one chunk at a time; the
        // partner wave holds the same lane position (the same sigma)
        if constexpr (W > 1) {
            __shared__ float xs[W][8][64];
#pragma unroll
            for (int j = 0; j < LOGW; ++j) {
                if (3 + LOGL + j < s0)
                    continue;
                const int pw = w ^ (1 << j);
                const float sw = ((w >> j) & 1) ? -1.0f : 1.0f;
#pragma unroll
                for (int cc = 0; cc < C; ++cc) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        xs[w][e][lane] = v[cc][e];
                    __syncthreads();
#pragma unroll
                    for (int e = 0; e < 8; ++e)  // u_lo + u_hi, or u_lo - u_hi
                        v[cc][e] = __builtin_fmaf(v[cc][e], sw, xs[pw][e][lane]);
                    __syncthreads();
                }
            }
        }
        // top bits: across the chunks of a lane
#pragma unroll
        for (int h = 1, bit = 3 + LOGL + LOGW; h < C; h <<= 1, ++bit)
            if (bit >= s0)
#pragma unroll
                for (int cc = 0; cc < C; ++cc)
                    if (!(cc & h)) {
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            float p = v[cc][e], q = v[cc + h][e];
                            v[cc][e] = p + q;
                            v[cc + h][e] = p - q;
                        }
                    }
        // y = u * c: sigma * c is exact and RN(sigma u * sigma c) = RN(u c).
        // The sign folding can leave -0 where the result is +0: the fp16 /
        // fp32 outputs take an fma with +0, which makes a zero +0; the
        // quantizers do not see the sign of a zero (|y|, y / s), except the
        // KV group bounds, which are made +0 once per group below.
        const float sc = sigma * a.c;
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if constexpr (EPI == EPI_F16 || EPI == EPI_F32)
                    v[cc][e] = __builtin_fmaf(v[cc][e], sc, 0.0f);
                else
                    v[cc][e] = v[cc][e] * sc;
            }
    }

    if constexpr (EPI == EPI_F16 || EPI == EPI_F32) {
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
            store_y8<EPI>(a.out, row * N + ((cc * W + w) * L + pos) * 8, v[cc]);
    } else if constexpr (EPI == EPI_SYM || EPI == EPI_SYM8 || EPI == EPI_E3M2) {
        __shared__ float red[W > 1 ? W : 1];
        float amax = 0.0f;
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                amax = fmaxf(amax, fabsf(v[cc][e]));
        amax = row_absmax<LOGL, W>(amax, w, red);
        const float qd = sym_divisor<EPI>(a);
        const float s32 = (amax * a.clip) / qd;
        const uint16_t s16 = f2h(s32);
        const Divisor dv = make_divisor(h2f(s16));
        if constexpr (EPI == EPI_E3M2) {
            // The codes as binary32 integers, four chunks (32 codes) at a
            // time through the fp6 pack conversion: its 192-bit result holds
            // code 2i of the first source and 2i + 1 of the second at bits
            // 12 i and 12 i + 6, so with chunk c's even codes at first-source
            // slots 4c .. 4c + 3 and its odd ones at the same second-source
            // slots, the chunk's 8 codes are bits 48 c .. 48 c + 47 in order.
            uint8_t *q6 = static_cast<uint8_t *>(a.out);
            // With 16 or more lanes per row a lane's 8 codes sit at the same
            // place p = pos mod 4 of unit (pos / 4) mod 4 of k-block
            // (c W + w) L / 16 + pos / 64 for chunk c: from chunk to chunk its
            // dword and short move by W L / 16 k-blocks.  (Shorter rows take
            // store_e3m2_48 per chunk.)
            constexpr bool STRIDED = L >= 16;
            uint8_t *dp = nullptr, *sp = nullptr;
            const int64_t kstep = (int64_t)(W * L / 16) * a.rows * 96;
            const bool podd = (pos & 1) != 0;
            if constexpr (STRIDED) {
                const int p = pos & 3, u = (pos >> 2) & 3, b0 = w * L / 16 + (pos >> 4);
                const int64_t h = e3m2_head(a.rows, row, b0, u), t = e3m2_tail(a.rows, row, b0, u);
                dp = q6 + (p == 0 ? h : p == 1 ? h + 8 : p == 2 ? h + 12 : t + 4);
                sp = q6 + (p == 0 ? h + 4 : p == 1 ? h + 6 : p == 2 ? t : t + 2);
            }
#pragma unroll
            for (int c0 = 0; c0 < C; c0 += 4) {
                v16f ev, od;
#pragma unroll
                for (int c = 0; c < 4 && c0 + c < C; ++c)
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float t = fminf(fmaxf(quotient(v[c0 + c][e], dv), -8.0f), 7.0f);
                        const float r = (t + 0x1.8p23f) - 0x1.8p23f;
                        if (e & 1)
                            od[4 * c + (e >> 1)] = r;
                        else
                            ev[4 * c + (e >> 1)] = r;
                    }
                v6i c6 = __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
                if (!dv.ok)  // zero or infinite scale: codes 0
                    c6 = v6i{0, 0, 0, 0, 0, 0};
#pragma unroll
                for (int c = 0; c < 4 && c0 + c < C; ++c) {
                    const int d = 3 * (c >> 1);  // first dword of the chunk pair
                    const uint32_t lo = (c & 1) ? __builtin_amdgcn_alignbit((uint32_t)c6[d + 2],
                                                                           (uint32_t)c6[d + 1], 16)
                                                : (uint32_t)c6[d];
                    const uint32_t hi = (c & 1) ? (uint32_t)c6[d + 2] >> 16
                                                : (uint32_t)c6[d + 1] & 0xFFFFu;
                    if constexpr (STRIDED) {
                        *reinterpret_cast<uint32_t *>(dp + (c0 + c) * kstep) =
                            podd ? (lo >> 16) | (hi << 16) : lo;
                        *reinterpret_cast<uint16_t *>(sp + (c0 + c) * kstep) =
                            (uint16_t)(podd ? lo : hi);
                    } else {
                        store_e3m2_48(q6, a.rows, row, ((c0 + c) * W + w) * L * 8 + pos * 8, lo,
                                      hi);
                    }
                }
            }
        } else {
            uint8_t *qr = static_cast<uint8_t *>(a.out) + row * sym_row_bytes<EPI>(N);
#pragma unroll
            for (int cc = 0; cc < C; ++cc)
                store_codes8<EPI>(qr, ((cc * W + w) * L + pos) * 8, v[cc], dv, qd);
        }
        if (pos == 0 && w == 0)
            a.scale[row] = s16;
    } else {  // EPI_KV: one wave per row; a group is G consecutive elements
        static_assert(W == 1, "KV rows fit one wave");
        // element i = (cc L + pos) 8 + e.  A group of G <= 8L elements is an
        // aligned block of G/8 positions of one chunk (lane_pos maps aligned
        // blocks of 2, 4, 8, 16 lanes onto themselves); a larger group takes
        // all L positions of G/(8L) consecutive chunks.
        const int gl = KVROW ? L * C : a.group >> 3;  // positions per group
        // chunk max and min as three-input max / min (v_max3 / v_min3: one
        // instruction per two values)
        float mx[C], mn[C];
        if constexpr (KVROW) {
            // the row is the group: the lane's chunks first, then its lanes
            float x = v[0][0], y = v[0][0];
#pragma unroll
            for (int cc = 0; cc < C; ++cc)
#pragma unroll
                for (int e = (cc == 0); e < 8; ++e) {
                    x = fmaxf(x, v[cc][e]);
                    y = fminf(y, v[cc][e]);
                }
            static_for<LOGL>([&](auto J) {
                if constexpr (J <= 1) {
                    dpp_maxmin<J>(x, y);
                } else {
                    x = lane_max<J>(x);
                    y = lane_min<J>(y);
                }
            });
#pragma unroll
            for (int cc = 0; cc < C; ++cc) {
                mx[cc] = x;
                mn[cc] = y;
            }
        } else {
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            const float *u = v[cc];
            mx[cc] = fmaxf(fmaxf(fmaxf(fmaxf(u[0], u[1]), u[2]), fmaxf(u[3], u[4])),
                           fmaxf(fmaxf(u[5], u[6]), u[7]));
            mn[cc] = fminf(fminf(fminf(fminf(u[0], u[1]), u[2]), fminf(u[3], u[4])),
                           fminf(fminf(u[5], u[6]), u[7]));
        }
        static_for<LOGL>([&](auto J) {
            if ((1 << J) < gl) {
                if constexpr (C == 4 && J <= 1) {
                    dpp_minmax4<J, true>(mx[0], mx[1], mx[2], mx[3]);
                    dpp_minmax4<J, false>(mn[0], mn[1], mn[2], mn[3]);
                } else {
#pragma unroll
                    for (int cc = 0; cc < C; ++cc) {
                        mx[cc] = lane_max<J>(mx[cc]);
                        mn[cc] = lane_min<J>(mn[cc]);
                    }
                }
            }
        });
#pragma unroll
        for (int h = 1; h < C; h <<= 1)
            if (h * L < gl) {
                float tx[C], tn[C];
#pragma unroll
                for (int cc = 0; cc < C; ++cc) {
                    tx[cc] = fmaxf(mx[cc], mx[cc ^ h]);
                    tn[cc] = fminf(mn[cc], mn[cc ^ h]);
                }
#pragma unroll
                for (int cc = 0; cc < C; ++cc) {
                    mx[cc] = tx[cc];
                    mn[cc] = tn[cc];
                }
            }
        }
        const int64_t orow = row * a.ostride + a.ooff;  // Append: a cache position
        uint8_t *qr = static_cast<uint8_t *>(a.out) + orow * (N / 2);
        uint16_t s16 = 0, z16 = 0;
        Divisor dv{};
        float zf = 0.0f;
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            // the group's scale and zero, formed again only where a group
            // starts (uniform across the wave)
            if (cc == 0 || (!KVROW && (cc * L) % gl == 0)) {
                // + 0: a bound that is a zero is +0 (see the rotation above)
                const float mxc = (mx[cc] + 0.0f) * a.clip, mnc = (mn[cc] + 0.0f) * a.clip;
                const float s32 = div15(mxc - mnc);
                s16 = f2h(s32);
                z16 = f2h(mnc);
                dv = make_divisor(h2f(s16));
                zf = h2f(z16);
            }
            // codes in the low nibbles of their rounding sums' encodings
            // (bits 4-15 of each are zero): pairs as bytes, bytes as
            // halves, then the two halves, one v_lshl_or_b32 per step (the
            // empty asm keeps the compiler from regrouping the ors)
            uint32_t f[8], p[4];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                f[e] = asym_code_bits(v[cc][e], dv, zf);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                p[k] = (f[2 * k + 1] << 4) | f[2 * k];
                __asm__("" : "+v"(p[k]));
            }
            const uint32_t lo = (p[1] << 8) | p[0], hi = (p[3] << 8) | p[2];
            const uint32_t pk = dv.ok ? perm_b32(hi, lo, 0x05040100u) : 0u;
            const int p8 = (cc * L + pos) * 8;  // first element of this chunk
            *reinterpret_cast<uint32_t *>(qr + p8 / 2) = pk;
            if (KVROW ? p8 == 0 : p8 % a.group == 0) {
                const int64_t gi = KVROW ? orow : orow * (N / a.group) + p8 / a.group;
                a.scale[gi] = s16;
                a.zero[gi] = z16;
            }
        }
    }
}

// ---------------------------------------------------- m = 12, 20, 28 -----

// The m-factor of one group of M fp16-valued inputs, exactly: each output
// u[b'] = RN32(sum_b H[b][b'] t[b]).  The sum runs in fp64, where every
// partial sum of fp16 values (multiples of 2^-24 below 2^21 in magnitude)
// is exact, so the order is free: inputs go in blocks of four (a, b, c, d),
// whose 8 signed sums a +- b +- c +- d cost 12 adds, and each output adds
// one signed block sum per block (the block's signs, normalised so that a
// enters with +, select which).  M = 28: 7 * 12 + 28 * 6 adds instead of
// 28 * 27.
template <int M>
__device__ __forceinline__ void mfactor_exact(float *t)
{
    static_assert(M % 4 == 0, "blocks of four");
    constexpr HmTable<M> H{};
    constexpr int G = M / 4;
    double acc[M];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const double a = t[4 * g], b = t[4 * g + 1], c = t[4 * g + 2], d = t[4 * g + 3];
        const double P[2] = {a + b, a - b}, Q[2] = {c + d, c - d};
        const double cp[2][2] = {{P[0] + Q[0], P[0] + Q[1]}, {P[1] + Q[0], P[1] + Q[1]}};
        const double cm[2][2] = {{P[0] - Q[0], P[0] - Q[1]}, {P[1] - Q[0], P[1] - Q[1]}};
#pragma unroll
        for (int bp = 0; bp < M; ++bp) {
            // contribution h0 a + h1 b + h2 c + h3 d
            //   = h0 ((a + h0h1 b) + h0h2 (c + h2h3 d))
            const float h0 = H.v[4 * g][bp], h1 = H.v[4 * g + 1][bp];
            const float h2 = H.v[4 * g + 2][bp], h3 = H.v[4 * g + 3][bp];
            const int i1 = (h0 * h1 < 0.0f), i3 = (h2 * h3 < 0.0f);
            const double blk = (h0 * h2 < 0.0f) ? cm[i1][i3] : cp[i1][i3];
            if (g == 0)
                acc[bp] = (h0 > 0.0f) ? blk : -blk;
            else
                acc[bp] = (h0 > 0.0f) ? acc[bp] + blk : acc[bp] - blk;
        }
    }
#pragma unroll
    for (int bp = 0; bp < M; ++bp)
        t[bp] = (float)acc[bp];  // the one rounding
}

template <int M, int LOGL, int W, int C, int EPI, int PRO = PRO_PLAIN>
__global__ __launch_bounds__(W == 1 ? 256 : 64 * W) void k_rot_smallm(RotArgs a)
{
    static_assert(M % 4 == 0, "groups load as 8-byte pieces");
    constexpr int L = 1 << LOGL;
    constexpr int LOGW = ilog2(W);
    constexpr int RPW = (W == 1) ? 64 / L : 1;
    constexpr int RPB = (W == 1) ? 4 * RPW : 1;
    constexpr int N = M * L * W * C;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pos = lane_pos(lane) & (L - 1);
    int64_t row;
    int w;
    if constexpr (W == 1) {
        row = (int64_t)blockIdx.x * RPB + wave * RPW + (lane >> LOGL);
        w = 0;
        if (row >= a.rows)
            return;
    } else {
        row = blockIdx.x;
        w = wave;
    }

    // LDS of the wave exchange below and, for fp16 output, of the row's
    // staging before its stores
    constexpr int XS_BYTES = W > 1 ? W * M * 64 * 4 : 16;
    constexpr int ST_BYTES = (EPI == EPI_F16 && W > 1) ? N * 2 : 16;
    __shared__ uint4 lbuf[(XS_BYTES > ST_BYTES ? XS_BYTES : ST_BYTES) / 16];

    float v[C][M];
#pragma unroll
    for (int cc = 0; cc < C; ++cc) {
        const int g = (cc * W + w) * L + pos;
#pragma unroll
        for (int p = 0; p < M / 4; ++p)
            load_row4<PRO>(a, row * N + g * M + 4 * p, &v[cc][4 * p]);
    }

#pragma unroll
    for (int cc = 0; cc < C; ++cc)
        mfactor_exact<M>(v[cc]);

    // group bits 0..LOGL-1 across lanes
    const float sigma = lane_stages<LOGL, C * M>(&v[0][0], lane, pos);
    if constexpr (W > 1) {
        float(*xs)[M][64] = reinterpret_cast<float(*)[M][64]>(lbuf);
#pragma unroll
        for (int j = 0; j < LOGW; ++j) {
            const int pw = w ^ (1 << j);
            const float sw = ((w >> j) & 1) ? -1.0f : 1.0f;
#pragma unroll
            for (int cc = 0; cc < C; ++cc) {
#pragma unroll
                for (int b = 0; b < M; ++b)
                    xs[w][b][lane] = v[cc][b];
                __syncthreads();
#pragma unroll
                for (int b = 0; b < M; ++b)
                    v[cc][b] = __builtin_fmaf(v[cc][b], sw, xs[pw][b][lane]);
                __syncthreads();
            }
        }
    }
#pragma unroll
    for (int h = 1; h < C; h <<= 1)
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
            if (!(cc & h)) {
#pragma unroll
                for (int b = 0; b < M; ++b) {
                    float p = v[cc][b], q = v[cc + h][b];
                    v[cc][b] = p + q;
                    v[cc + h][b] = p - q;
                }
            }
    const float sc = sigma * a.c;  // as in k_rot_pow2: +0 zeros where the sign shows
#pragma unroll
    for (int cc = 0; cc < C; ++cc)
#pragma unroll
        for (int b = 0; b < M; ++b) {
            if constexpr (EPI == EPI_F16 || EPI == EPI_F32)
                v[cc][b] = __builtin_fmaf(v[cc][b], sc, 0.0f);
            else
                v[cc][b] = v[cc][b] * sc;
        }

    if constexpr (EPI == EPI_F16 && W > 1) {
        // a lane's M outputs sit 2 M bytes apart from the next lane's: the
        // row goes through LDS (the exchange's, whose last reads are behind
        // its barriers) and out as 16 consecutive bytes per lane
        uint16_t *st = reinterpret_cast<uint16_t *>(lbuf);
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            const int g = (cc * W + w) * L + pos;
#pragma unroll
            for (int p = 0; p < M / 4; ++p)
                store4(st + g * M + 4 * p, &v[cc][4 * p]);
        }
        __syncthreads();
        uint4 *dst = reinterpret_cast<uint4 *>(static_cast<uint16_t *>(a.out) + row * N);
        for (int c = tid; c < N / 8; c += 64 * W)
            dst[c] = lbuf[c];
    } else if constexpr (EPI == EPI_F32 && W > 1) {
        // the same for binary32 output, one chunk cc (W L groups, M W L
        // consecutive elements, the size of the exchange's buffer) at a time
        float *st = reinterpret_cast<float *>(lbuf);
        static_assert(M * W * 64 * 4 <= XS_BYTES, "a chunk fits the exchange buffer");
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            const int g = w * L + pos;  // group within the chunk
#pragma unroll
            for (int p = 0; p < M / 4; ++p)
                *reinterpret_cast<float4 *>(st + g * M + 4 * p) =
                    make_float4(v[cc][4 * p], v[cc][4 * p + 1], v[cc][4 * p + 2], v[cc][4 * p + 3]);
            __syncthreads();
            uint4 *dst = reinterpret_cast<uint4 *>(static_cast<float *>(a.out) + row * N +
                                                   (int64_t)cc * (M * W * L));
            for (int c = tid; c < M * W * L / 4; c += 64 * W)
                dst[c] = lbuf[c];
            __syncthreads();
        }
    } else if constexpr (EPI == EPI_F16 || EPI == EPI_F32) {
#pragma unroll
        for (int cc = 0; cc < C; ++cc) {
            const int g = (cc * W + w) * L + pos;
#pragma unroll
            for (int p = 0; p < M / 4; ++p)
                store_y4<EPI>(a.out, row * N + g * M + 4 * p, &v[cc][4 * p]);
        }
    } else {
        static_assert(EPI == EPI_SYM || EPI == EPI_SYM8 || EPI == EPI_E3M2,
                      "small-m kernels serve activations");
        static_assert(EPI != EPI_E3M2 || W > 1, "e3m2 rows stage in LDS: one row per block");
        __shared__ float red[W > 1 ? W : 1];
        float amax = 0.0f;
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
#pragma unroll
            for (int b = 0; b < M; ++b)
                amax = fmaxf(amax, fabsf(v[cc][b]));
        amax = row_absmax<LOGL, W>(amax, w, red);
        const float qd = sym_divisor<EPI>(a);
        const float s32 = (amax * a.clip) / qd;
        const uint16_t s16 = f2h(s32);
        const Divisor dv = make_divisor(h2f(s16));
        if constexpr (EPI == EPI_E3M2) {
            // a lane's M codes do not fill whole 32-code units: the row's
            // codes go through LDS as signed bytes (the EPI_SYM decision:
            // clamp to -8..7, ties to even; 0 for a zero or infinite scale),
            // then each thread takes whole units: 32 bytes back to binary32
            // and one fp6 pack conversion (code 2i from slot i of the first
            // source, 2i + 1 from slot i of the second)
            __shared__ uint4 stage[N / 16];
            uint8_t *st = reinterpret_cast<uint8_t *>(stage);
#pragma unroll
            for (int cc = 0; cc < C; ++cc) {
                const int g = (cc * W + w) * L + pos;
#pragma unroll
                for (int p = 0; p < M / 4; ++p)
                    store_codes4<EPI_SYM8>(st, g * M + 4 * p, &v[cc][4 * p], dv, 7.0f);
            }
            __syncthreads();
            uint8_t *q = static_cast<uint8_t *>(a.out);
            for (int u = tid; u < N / 32; u += 64 * W) {
                const uint4 in0 = stage[2 * u], in1 = stage[2 * u + 1];
                const uint32_t wd[8] = {in0.x, in0.y, in0.z, in0.w, in1.x, in1.y, in1.z, in1.w};
                v16f ev, od;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    ev[2 * k] = (float)(int8_t)(wd[k] & 0xFFu);
                    od[2 * k] = (float)(int8_t)((wd[k] >> 8) & 0xFFu);
                    ev[2 * k + 1] = (float)(int8_t)((wd[k] >> 16) & 0xFFu);
                    od[2 * k + 1] = (float)(int8_t)(wd[k] >> 24);
                }
                const v6i o = __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
                *reinterpret_cast<uint4 *>(q + e3m2_head(a.rows, row, u >> 2, u & 3)) =
                    make_uint4((uint32_t)o[0], (uint32_t)o[1], (uint32_t)o[2], (uint32_t)o[3]);
                *reinterpret_cast<uint2 *>(q + e3m2_tail(a.rows, row, u >> 2, u & 3)) =
                    make_uint2((uint32_t)o[4], (uint32_t)o[5]);
            }
        } else {
            uint8_t *qr = static_cast<uint8_t *>(a.out) + row * sym_row_bytes<EPI>(N);
#pragma unroll
            for (int cc = 0; cc < C; ++cc) {
                const int g = (cc * W + w) * L + pos;
#pragma unroll
                for (int p = 0; p < M / 4; ++p)
                    store_codes4<EPI>(qr, g * M + 4 * p, &v[cc][4 * p], dv, qd);
            }
        }
        if (pos == 0 && w == 0)
            a.scale[row] = s16;
    }
}

// ------------------------------------------------------- m = 108, 172 -----

template <int M>
__device__ __forceinline__ const uint4 *hm_mfma_b();
template <>
__device__ __forceinline__ const uint4 *hm_mfma_b<108>()
{
    return reinterpret_cast<const uint4 *>(&c_hmb108.w[0][0][0][0]);
}
template <>
__device__ __forceinline__ const uint4 *hm_mfma_b<172>()
{
    return reinterpret_cast<const uint4 *>(&c_hmb172.w[0][0][0][0]);
}

// Four fp16 inputs (raw bits) at element offset off of the row: the plain
// row, or RN16(silu(gate) up) for the SwiGLU prologue.
template <int PRO>
__device__ __forceinline__ uint2 load_bits4(const RotArgs &a, int64_t off)
{
    if constexpr (PRO == PRO_PLAIN) {
        return *reinterpret_cast<const uint2 *>(a.x + off);
    } else {
        float v[4];
        load_row4<PRO>(a, off, v);
        return make_uint2((uint32_t)f2h(v[0]) | ((uint32_t)f2h(v[1]) << 16),
                          (uint32_t)f2h(v[2]) | ((uint32_t)f2h(v[3]) << 16));
    }
}

// One row per block of four waves; the row's A = n / M groups of M
// elements (element i = g M + b).
//
// m-factor on the int8 matrix cores.  It is a contraction, U = T . H_M
// with T [A, M] the groups: every fp16 input is an integer multiple of
// 2^-24, so N = t 2^24 is an integer below 2^40, and its signed base-64
// digits (f16_planes) are int8 operands of v_mfma_i32_16x16x64_i8 against
// the +-1 entries of H_M.  Digits 2p and 2p+1 accumulate into one int32 C_p
// (the odd digit against 64 H_M, still int8): |C_p| <= M * 63 * 65 < 2^21.
// Then
// sum_b H[b][b'] N_b = sum_p C_p 2^(12 p), an integer below 2^48, is formed
// exactly in binary64 and u = RN32(that * 2^-24): the exact sum rounded
// once, as the definition asks, in whatever order the hardware adds.
//
// A wave takes row tiles of 16 groups (groups past A are zero); the MFMA
// output puts groups 4 (l/16) + r (register r) and column ct*16 + l%16 in
// lane l, so Walsh-Hadamard bits 0-1 of the group index are butterflies
// between registers and bits 2-3 between lanes l and l ^ 16, l ^ 32; u is
// then staged in LDS as the row itself (element i = g M + b at i).  Bits
// 4.. (across tiles) run in registers on the 2^(k-4) values of one column
// of the groups a, a + 16, ..., which also gives the row's absmax; the
// epilogue reads 8 consecutive elements with two 16-byte reads.  H_M's
// operand tiles sit in LDS in front of the row.
template <int M, int EPI, int PRO = PRO_PLAIN>
__global__ __launch_bounds__(256, 2) void k_rot_largem(RotArgs a)
{
    constexpr int W = 4;
    constexpr int CT = HmMfmaB<M>::CT, KB = HmMfmaB<M>::KB;
    constexpr int CTP = 4;  // column tiles per pass (accumulator registers)
    static_assert(M % 4 == 0, "4-element loads");
    typedef int v4i __attribute__((ext_vector_type(4)));
    extern __shared__ __align__(16) uint8_t lds_raw[];
    uint4 *hb = reinterpret_cast<uint4 *>(lds_raw);                 // [CT][KB][64]
    float *rowbuf = reinterpret_cast<float *>(lds_raw + CT * KB * 1024);
    __shared__ float red[W];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = a.n, A = n / M;
    const int k = 31 - __clz(A);
    const int64_t row = blockIdx.x;

    {
        const uint4 *src = hm_mfma_b<M>();
        for (int i = tid; i < CT * KB * 64; i += 64 * W)
            hb[i] = src[i];
    }
    __syncthreads();

    const int RT = A >= 16 ? A / 16 : 1;  // row tiles of 16 groups
    const int kreg = k < 4 ? k : 4;       // group bits done in registers / lanes
    for (int rt = wave; rt < RT; rt += W) {
        // A operands: digit d of the 16 inputs b = kb*64 + (lane/16)*16 + e
        // of group rt*16 + lane%16, byte e (zeros past the row or the group)
        const int g = rt * 16 + (lane & 15);
        v4i dig[KB][7];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            uint32_t w[7][4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                // past the row or the group: load a valid quad, use zeros
                const int b = kb * 64 + (lane >> 4) * 16 + 4 * q;
                const bool ok = g < A && b < M;
                const uint2 ld = load_bits4<PRO>(
                    a, row * n + (int64_t)(ok ? g : 0) * M + (ok ? b : 0));
                const uint2 raw = ok ? ld : make_uint2(0, 0);
                uint32_t d[7];
                f16x4_planes(raw, d);
#pragma unroll
                for (int i = 0; i < 7; ++i)
                    w[i][q] = d[i];
            }
#pragma unroll
            for (int i = 0; i < 7; ++i)
                dig[kb][i] = v4i{(int)w[i][0], (int)w[i][1], (int)w[i][2], (int)w[i][3]};
        }
#pragma unroll
        for (int c0 = 0; c0 < CT; c0 += CTP) {
            v4i acc[CTP][4];
#pragma unroll
            for (int c = 0; c < CTP; ++c)
#pragma unroll
                for (int p = 0; p < 4; ++p)
                    acc[c][p] = v4i{0, 0, 0, 0};
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int c = 0; c < CTP; ++c) {
                    if (c0 + c >= CT)
                        continue;
                    const uint4 hv = hb[((c0 + c) * KB + kb) * 64 + lane];
                    // 64 H: each byte +-1 -> +-64 (bytes hold -1 as 0xFF, so
                    // shifting the dword left by 6 and keeping bits 6-7 of
                    // every byte gives 0xC0 / 0x40 with no carry between bytes)
                    const v4i h1 = v4i{(int)hv.x, (int)hv.y, (int)hv.z, (int)hv.w};
                    const v4i h64 = v4i{(int)((hv.x << 6) & 0xC0C0C0C0u), (int)((hv.y << 6) & 0xC0C0C0C0u),
                                        (int)((hv.z << 6) & 0xC0C0C0C0u), (int)((hv.w << 6) & 0xC0C0C0C0u)};
#pragma unroll
                    for (int i = 0; i < 7; ++i)
                        acc[c][i >> 1] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                            dig[kb][i], (i & 1) ? h64 : h1, acc[c][i >> 1], 0, 0, 0);
                }
#pragma unroll
            for (int c = 0; c < CTP; ++c) {
                if (c0 + c >= CT)
                    continue;
                float u[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    double x = (double)acc[c][3][r];
                    x = __builtin_fma(x, 4096.0, (double)acc[c][2][r]);
                    x = __builtin_fma(x, 4096.0, (double)acc[c][1][r]);
                    x = __builtin_fma(x, 4096.0, (double)acc[c][0][r]);
                    u[r] = (float)(x * 0x1p-24);  // exact scaling, one rounding
                }
                // Walsh-Hadamard bits 0..kreg-1 of the group index, bit 0
                // first: registers (bits 0, 1), then lanes (bits 2, 3)
                if (kreg > 0) {
                    const float p0 = u[0], p2 = u[2];
                    u[0] = p0 + u[1];
                    u[1] = p0 - u[1];
                    u[2] = p2 + u[3];
                    u[3] = p2 - u[3];
                }
                if (kreg > 1) {
                    const float p0 = u[0], p1 = u[1];
                    u[0] = p0 + u[2];
                    u[1] = p1 + u[3];
                    u[2] = p0 - u[2];
                    u[3] = p1 - u[3];
                }
#pragma unroll
                for (int j = 2; j < 4; ++j) {
                    if (kreg > j) {
                        const int mask = 16 << (j - 2);
                        const bool hi = (lane & mask) != 0;
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float o = __shfl_xor(u[r], mask);
                            u[r] = hi ? o - u[r] : u[r] + o;
                        }
                    }
                }
                const int col = (c0 + c) * 16 + (lane & 15);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int gg = rt * 16 + 4 * (lane >> 4) + r;
                    if (gg < A && col < M)
                        rowbuf[gg * M + col] = u[r];
                }
            }
        }
    }
    __syncthreads();
    // group bits 4.. (across row tiles) and the row's absmax: a thread takes
    // column b of the groups a, a + 16, ... (a < 16), their 2^(k-4) values
    const float c = a.c;
    float amax = 0.0f;
    auto column_pass = [&](auto NJ_) {
        constexpr int NJ = decltype(NJ_)::value;
        const int NA = NJ > 1 ? 16 : A;
        for (int idx = tid; idx < NA * M; idx += 64 * W) {
            const int al = idx / M, b = idx - al * M;
            float v[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                v[j] = rowbuf[(al + 16 * j) * M + b];
#pragma unroll
            for (int h = 1; h < NJ; h <<= 1)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    if (!(j & h)) {
                        const float p = v[j], q = v[j + h];
                        v[j] = p + q;
                        v[j + h] = p - q;
                    }
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                if constexpr (NJ > 1)
                    rowbuf[(al + 16 * j) * M + b] = v[j];
                amax = fmaxf(amax, fabsf(v[j] * c));  // |y|: the sign of a zero is moot
            }
        }
    };
    switch (k) {
    case 7: column_pass(std::integral_constant<int, 8>()); break;
    case 6: column_pass(std::integral_constant<int, 4>()); break;
    case 5: column_pass(std::integral_constant<int, 2>()); break;
    default: column_pass(std::integral_constant<int, 1>()); break;
    }
    __syncthreads();
    const int chunks = n / 8;
    auto row8 = [&](int ch, float *y) {
        const float4 p0 = *reinterpret_cast<const float4 *>(rowbuf + ch * 8);
        const float4 p1 = *reinterpret_cast<const float4 *>(rowbuf + ch * 8 + 4);
        y[0] = p0.x, y[1] = p0.y, y[2] = p0.z, y[3] = p0.w;
        y[4] = p1.x, y[5] = p1.y, y[6] = p1.z, y[7] = p1.w;
    };
    if constexpr (EPI == EPI_F16 || EPI == EPI_F32) {
        for (int ch = tid; ch < chunks; ch += 64 * W) {
            float y[8];
            row8(ch, y);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                y[e] = __builtin_fmaf(y[e], c, 0.0f);  // zeros +0
            store_y8<EPI>(a.out, row * n + ch * 8, y);
        }
    } else {
        static_assert(EPI == EPI_SYM || EPI == EPI_SYM8 || EPI == EPI_E3M2,
                      "large-m kernels serve activations");
        static_for<6>([&](auto J) { amax = lane_max<J>(amax); });
        if (lane == 0)
            red[tid >> 6] = amax;
        __syncthreads();
        amax = red[0];
#pragma unroll
        for (int i = 1; i < W; ++i)
            amax = fmaxf(amax, red[i]);
        const float qd = sym_divisor<EPI>(a);
        const float s32 = (amax * a.clip) / qd;
        const uint16_t s16 = f2h(s32);
        const Divisor dv = make_divisor(h2f(s16));
        if constexpr (EPI == EPI_E3M2) {
            // a thread takes whole units (32 consecutive codes) through one
            // fp6 pack conversion (code 2i from slot i of the first source,
            // 2i + 1 from slot i of the second)
            uint8_t *q6 = static_cast<uint8_t *>(a.out);
            for (int u = tid; u < chunks / 4; u += 64 * W) {
                v16f ev, od;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    float y[8];
                    row8(4 * u + k, y);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float t = fminf(fmaxf(quotient(y[e] * c, dv), -8.0f), 7.0f);
                        const float r = (t + 0x1.8p23f) - 0x1.8p23f;
                        if (e & 1)
                            od[4 * k + (e >> 1)] = r;
                        else
                            ev[4 * k + (e >> 1)] = r;
                    }
                }
                v6i o = __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
                if (!dv.ok)  // zero or infinite scale: codes 0
                    o = v6i{0, 0, 0, 0, 0, 0};
                *reinterpret_cast<uint4 *>(q6 + e3m2_head(a.rows, row, u >> 2, u & 3)) =
                    make_uint4((uint32_t)o[0], (uint32_t)o[1], (uint32_t)o[2], (uint32_t)o[3]);
                *reinterpret_cast<uint2 *>(q6 + e3m2_tail(a.rows, row, u >> 2, u & 3)) =
                    make_uint2((uint32_t)o[4], (uint32_t)o[5]);
            }
        } else {
            uint8_t *qr = static_cast<uint8_t *>(a.out) + row * sym_row_bytes<EPI>(n);
            for (int ch = tid; ch < chunks; ch += 64 * W) {
                float y[8];
                row8(ch, y);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    y[e] = y[e] * c;
                store_codes8<EPI>(qr, ch * 8, y, dv, qd);
            }
        }
        if (tid == 0)
            a.scale[row] = s16;
    }
}

// ------------------------------------------------- no rotation, any n -----

template <int EPI>
__global__ __launch_bounds__(256) void k_quant_plain(RotArgs a)
{
    __shared__ float red[4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t row = blockIdx.x;
    const int n = a.n, chunks = n / 8;
    const uint16_t *xr = a.x + row * n;
    float amax = 0.0f;
    for (int ch = tid; ch < chunks; ch += 256) {
        float v[8];
        load8(xr + ch * 8, v);
#pragma unroll
        for (int e = 0; e < 8; ++e)
            amax = fmaxf(amax, fabsf(v[e]));
    }
    static_for<6>([&](auto J) { amax = lane_max<J>(amax); });
    if (lane == 0)
        red[tid >> 6] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const float qd = sym_divisor<EPI>(a);
    const float s32 = (amax * a.clip) / qd;
    const uint16_t s16 = f2h(s32);
    const Divisor dv = make_divisor(h2f(s16));
    if constexpr (EPI == EPI_E3M2) {
        // whole units through one fp6 pack conversion, as in k_rot_largem
        uint8_t *q6 = static_cast<uint8_t *>(a.out);
        for (int u = tid; u < chunks / 4; u += 256) {
            v16f ev, od;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                float v[8];
                load8(xr + (4 * u + k) * 8, v);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float t = fminf(fmaxf(quotient(v[e], dv), -8.0f), 7.0f);
                    const float r = (t + 0x1.8p23f) - 0x1.8p23f;
                    if (e & 1)
                        od[4 * k + (e >> 1)] = r;
                    else
                        ev[4 * k + (e >> 1)] = r;
                }
            }
            v6i o = __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
            if (!dv.ok)  // zero or infinite scale: codes 0
                o = v6i{0, 0, 0, 0, 0, 0};
            *reinterpret_cast<uint4 *>(q6 + e3m2_head(a.rows, row, u >> 2, u & 3)) =
                make_uint4((uint32_t)o[0], (uint32_t)o[1], (uint32_t)o[2], (uint32_t)o[3]);
            *reinterpret_cast<uint2 *>(q6 + e3m2_tail(a.rows, row, u >> 2, u & 3)) =
                make_uint2((uint32_t)o[4], (uint32_t)o[5]);
        }
    } else {
        uint8_t *qr = static_cast<uint8_t *>(a.out) + row * sym_row_bytes<EPI>(n);
        for (int ch = tid; ch < chunks; ch += 256) {
            float v[8];
            load8(xr + ch * 8, v);
            store_codes8<EPI>(qr, ch * 8, v, dv, qd);
        }
    }
    if (tid == 0)
        a.scale[row] = s16;
}

// ------------------------------------------------- elementwise SwiGLU -----

// h = RN16(RN(silu(gate) up)), 8 elements per thread and step.
__global__ __launch_bounds__(256) void k_swiglu(const uint16_t *g, const uint16_t *u,
                                                uint16_t *h, int64_t chunks)
{
    RotArgs a{};
    a.x = g;
    a.x2 = u;
    for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < chunks;
         c += (int64_t)gridDim.x * 256) {
        float v[8];
        load_row8<PRO_SWIGLU>(a, c * 8, v);
        store8(h + c * 8, v);  // exact: v holds fp16 values
    }
}

// ------------------------------------------------ weights' clip search ---

// Per-row clip search (§5 Setup: the weights' clipping ratio by a linear
// search over the squared error; App. A.2).  One block per row.  For each
// candidate c_j = RN32((100 - j) / 100) the symmetric quantizer's scale and
// codes, and E_j = sum RN64((y - q s16)^2) with each difference exact in
// binary64, summed in a fixed order (256 interleaved partial sums, then a
// halving tree; see below).  The row keeps the first j with the smallest
// E_j, then writes its codes, scale and clip.
template <int BITS, typename TIN>
__global__ __launch_bounds__(256) void k_quant_search(SearchArgs a)
{
    constexpr int QMAX = BITS == 4 ? 7 : BITS == 6 ? 31 : 127;
    constexpr float QF = (float)QMAX;
    __shared__ float redf[4];
    __shared__ double redd[256];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const int n = a.n, chunks = n / 8;
    const TIN *yr = static_cast<const TIN *>(a.y) + row * n;
    auto load = [&](int ch, float *v) {
        if constexpr (sizeof(TIN) == 4) {
            const float4 p0 = reinterpret_cast<const float4 *>(yr + ch * 8)[0];
            const float4 p1 = reinterpret_cast<const float4 *>(yr + ch * 8)[1];
            v[0] = p0.x, v[1] = p0.y, v[2] = p0.z, v[3] = p0.w;
            v[4] = p1.x, v[5] = p1.y, v[6] = p1.z, v[7] = p1.w;
        } else {
            load8(reinterpret_cast<const uint16_t *>(yr) + ch * 8, v);
        }
    };
    float amax = 0.0f;
    for (int ch = tid; ch < chunks; ch += 256) {
        float v[8];
        load(ch, v);
#pragma unroll
        for (int e = 0; e < 8; ++e)
            amax = fmaxf(amax, fabsf(v[e]));
    }
    static_for<6>([&](auto J) { amax = lane_max<J>(amax); });
    if (lane == 0)
        redf[wave] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(redf[0], redf[1]), fmaxf(redf[2], redf[3]));

    double best_e = __builtin_inf();
    float best_c = 1.0f;
    for (int j = 0; j < a.ncand; ++j) {
        const float c = (float)((double)(100 - j) / 100.0);
        const float sf = h2f(f2h((amax * c) / QF));
        const Divisor dv = make_divisor(sf);
        // The error's defined binary64 order: thread t sums the terms of
        // elements t, t + 256, ... from +0 in increasing index; the 256
        // partial sums P_t are then halved pairwise (P_t += P_{t+h},
        // h = 128, ..., 1).  Every wave evaluates the whole tree from the
        // LDS copy, so all threads hold the same total.
        double e = 0.0;
        for (int i = tid; i < n; i += 256) {
            float v;
            if constexpr (sizeof(TIN) == 4)
                v = yr[i];
            else
                v = h2f(yr[i]);  // fp16 bits
            const float cq = dv.ok ? fminf(fmaxf(rintf(quotient(v, dv)), -QF - 1.0f), QF)
                                   : 0.0f;
            const double d = (double)v - (double)cq * (double)sf;
            const double t = d * d;  // rounded on its own (no contraction)
            e = e + t;
        }
        __syncthreads();  // redd of the previous candidate has been read
        redd[tid] = e;
        __syncthreads();
        // h = 128 and h = 64: lane l of any wave forms
        // (P_l + P_{l+128}) + (P_{l+64} + P_{l+192})
        e = (redd[lane] + redd[lane + 128]) + (redd[lane + 64] + redd[lane + 192]);
        // h = 32 .. 1: the xor butterflies give lane l the sum of lanes l
        // and l ^ h, which for l < h is the tree's P_l + P_{l+h}
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1)
            e = e + __shfl_xor(e, o);
        if (e < best_e) {  // uniform across the block
            best_e = e;
            best_c = c;
        }
    }
    const uint16_t s16 = f2h((amax * best_c) / QF);
    const Divisor dv = make_divisor(h2f(s16));
    uint8_t *qr = static_cast<uint8_t *>(a.q) + row * (BITS == 4 ? n / 2 : n);
    for (int ch = tid; ch < chunks; ch += 256) {
        float v[8];
        load(ch, v);
        if constexpr (BITS == 4)
            store_codes8<EPI_SYM>(qr, ch * 8, v, dv, QF);
        else
            store_codes8<EPI_SYM8>(qr, ch * 8, v, dv, QF);
    }
    if (tid == 0) {
        a.scale[row] = s16;
        a.clip[row] = best_c;
    }
}

// --------------------------------------------- group-wise quantization ---

// Group-wise symmetric int4 (§5.3 group-wise ablation): every G = 8 L
// consecutive elements of a row get their own absmax, fp16 scale and codes,
// exactly as a whole row does per token.  L lanes hold one group (8
// elements each) and reduce its absmax among themselves; a block of 256
// threads covers one group column g of 256 / L consecutive rows, so the
// group-major scale writes s[g][r0 ..] are contiguous.
template <int LOGL, typename TIN>
__global__ __launch_bounds__(256) void k_quant_grouped(const void *y, uint8_t *q,
                                                       uint16_t *scale, int64_t rows, int n,
                                                       float clip)
{
    constexpr int L = 1 << LOGL, G = 8 * L, R = 256 / L;
    const int ng = n / G;
    const int g = (int)(blockIdx.x % (unsigned)ng);
    const int64_t row = (int64_t)(blockIdx.x / (unsigned)ng) * R + (threadIdx.x >> LOGL);
    const int li = threadIdx.x & (L - 1);
    if (row >= rows)  // a whole group of lanes leaves together
        return;
    const int64_t e0 = row * n + (int64_t)g * G + li * 8;
    float v[8];
    if constexpr (sizeof(TIN) == 4) {
        const float4 p0 = reinterpret_cast<const float4 *>(static_cast<const float *>(y) + e0)[0];
        const float4 p1 = reinterpret_cast<const float4 *>(static_cast<const float *>(y) + e0)[1];
        v[0] = p0.x, v[1] = p0.y, v[2] = p0.z, v[3] = p0.w;
        v[4] = p1.x, v[5] = p1.y, v[6] = p1.z, v[7] = p1.w;
    } else {
        load8(static_cast<const uint16_t *>(y) + e0, v);
    }
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e)
        amax = fmaxf(amax, fabsf(v[e]));
    static_for<LOGL>([&](auto J) { amax = lane_max<J>(amax); });
    const uint16_t s16 = f2h((amax * clip) / 7.0f);
    const Divisor dv = make_divisor(h2f(s16));
    store_codes8<EPI_SYM>(q, e0, v, dv, 7.0f);
    if (li == 0)
        scale[(int64_t)g * rows + row] = s16;
}

// ------------------------------------------------------ KV dequant -------

template <int LOGL, int C, bool INV>
__global__ __launch_bounds__(256) void k_kv_dequant(KvDeqArgs a)
{
    constexpr int L = 1 << LOGL;
    constexpr int RPW = 64 / L, RPB = 4 * RPW, N = 8 * L * C;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pos = lane_pos(lane) & (L - 1);
    const int64_t row = (int64_t)blockIdx.x * RPB + wave * RPW + (lane >> LOGL);
    if (row >= a.rows)
        return;
    float v[C][8];
#pragma unroll
    for (int cc = 0; cc < C; ++cc) {
        const int p8 = (cc * L + pos) * 8;  // element index i = (cc L + pos) 8 + e
        const uint32_t pk = *reinterpret_cast<const uint32_t *>(a.q + row * (N / 2) + p8 / 2);
        const int64_t gi = row * (N / a.group) + p8 / a.group;
        const float sf = h2f(a.scale[gi]), zf = h2f(a.zero[gi]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float t = (float)((pk >> (4 * e)) & 0xFu) * sf;
            v[cc][e] = t + zf;
        }
    }
    if constexpr (INV) {
#pragma unroll
        for (int h = 1; h < 8; h <<= 1)
#pragma unroll
            for (int cc = 0; cc < C; ++cc)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (!(e & h)) {
                        float p = v[cc][e], q = v[cc][e + h];
                        v[cc][e] = p + q;
                        v[cc][e + h] = p - q;
                    }
        const float sc = lane_stages<LOGL, 8 * C>(&v[0][0], lane, pos) * a.c;
#pragma unroll
        for (int h = 1; h < C; h <<= 1)
#pragma unroll
            for (int cc = 0; cc < C; ++cc)
                if (!(cc & h)) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        float p = v[cc][e], q = v[cc + h][e];
                        v[cc][e] = p + q;
                        v[cc + h][e] = p - q;
                    }
                }
#pragma unroll
        for (int cc = 0; cc < C; ++cc)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[cc][e] = __builtin_fmaf(v[cc][e], sc, 0.0f);  // zeros +0, as in k_rot_pow2
    }
#pragma unroll
    for (int cc = 0; cc < C; ++cc)
        store8(a.out + row * N + (cc * L + pos) * 8, v[cc]);
}

// ---------------------------------------------------------- dispatch -----

template <int LOGL, int W, int C, int EPI, bool ROT, int PRO, bool HEADS, bool KVROW>
hipError_t go_pow2(const RotArgs &a, hipStream_t s)
{
    constexpr int L = 1 << LOGL;
    constexpr int RPB = (W == 1) ? 4 * (64 / L) : 1;
    const int64_t blocks = (a.rows + RPB - 1) / RPB;
    hipLaunchKernelGGL((k_rot_pow2<LOGL, W, C, EPI, ROT, PRO, HEADS, KVROW>),
                       dim3((unsigned)blocks), dim3(W == 1 ? 256 : 64 * W), 0, s, a);
    return hipGetLastError();
}

template <int M, int LOGL, int W, int C, int EPI, int PRO>
hipError_t go_smallm(const RotArgs &a, hipStream_t s)
{
    constexpr int L = 1 << LOGL;
    constexpr int RPB = (W == 1) ? 4 * (64 / L) : 1;
    const int64_t blocks = (a.rows + RPB - 1) / RPB;
    hipLaunchKernelGGL((k_rot_smallm<M, LOGL, W, C, EPI, PRO>), dim3((unsigned)blocks),
                       dim3(W == 1 ? 256 : 64 * W), 0, s, a);
    return hipGetLastError();
}

template <int M, int EPI, int PRO>
hipError_t go_largem(const RotArgs &a, hipStream_t s)
{
    // H_M's operand tiles, then the staged row
    const size_t lds = (size_t)HmMfmaB<M>::CT * HmMfmaB<M>::KB * 1024 +
                       (size_t)a.n * sizeof(float);
    const void *fn = (const void *)k_rot_largem<M, EPI, PRO>;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((k_rot_largem<M, EPI, PRO>), dim3((unsigned)a.rows), dim3(256), lds, s, a);
    return hipGetLastError();
}

template <int EPI, bool ROT, int PRO, bool HEADS = false, bool KVROW = false>
hipError_t dispatch_pow2(const RotArgs &a, int k, hipStream_t s)
{
    // short rows: up to 4 chunks (32 elements) per lane, D / 32 lanes per row
    switch (k) {
    case 3: return go_pow2<0, 1, 1, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 4: return go_pow2<0, 1, 2, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 5: return go_pow2<0, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 6: return go_pow2<1, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 7: return go_pow2<2, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 8: return go_pow2<3, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    case 9: return go_pow2<4, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
    }
    if constexpr (EPI != EPI_KV) {
        switch (k) {
        case 10: return go_pow2<6, 1, 2, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        case 11: return go_pow2<6, 1, 4, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        case 12: return go_pow2<6, 1, 8, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        case 13: return go_pow2<6, 2, 8, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        case 14: return go_pow2<6, 4, 8, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        case 15: return go_pow2<6, 8, 8, EPI, ROT, PRO, HEADS, KVROW>(a, s);
        }
    }
    return hipErrorInvalidValue;
}

// groups A = 2^k; C = min(A/64, CMAX) chunks per lane, W = A/(64 C) waves
template <int M, int CMAX, int EPI, int PRO>
hipError_t dispatch_smallm(const RotArgs &a, int k, hipStream_t s)
{
    switch (k) {
    case 0: return go_smallm<M, 0, 1, 1, EPI, PRO>(a, s);
    case 1: return go_smallm<M, 1, 1, 1, EPI, PRO>(a, s);
    case 2: return go_smallm<M, 2, 1, 1, EPI, PRO>(a, s);
    case 3: return go_smallm<M, 3, 1, 1, EPI, PRO>(a, s);
    case 4: return go_smallm<M, 4, 1, 1, EPI, PRO>(a, s);
    case 5: return go_smallm<M, 5, 1, 1, EPI, PRO>(a, s);
    case 6: return go_smallm<M, 6, 1, 1, EPI, PRO>(a, s);
    case 7: return go_smallm<M, 6, 1, 2, EPI, PRO>(a, s);
    case 8: return go_smallm<M, 6, 1, 4, EPI, PRO>(a, s);
    case 9: return go_smallm<M, 6, (CMAX >= 8 ? 1 : 2), (CMAX >= 8 ? 8 : 4), EPI, PRO>(a, s);
    case 10: return go_smallm<M, 6, (CMAX >= 8 ? 2 : 4), (CMAX >= 8 ? 8 : 4), EPI, PRO>(a, s);
    case 11:
        if constexpr (CMAX >= 8)
            return go_smallm<M, 6, 4, 8, EPI, PRO>(a, s);
        break;
    }
    return hipErrorInvalidValue;
}

// e3m2 output from the small-m kernels: the configurations with one row per
// block (the row is staged in LDS)
template <int M, int PRO>
hipError_t dispatch_smallm_e3m2(const RotArgs &a, int k, hipStream_t s)
{
    if constexpr (M == 12) {
        if (k == 10)
            return go_smallm<12, 6, 2, 8, EPI_E3M2, PRO>(a, s);
        if (k == 11)
            return go_smallm<12, 6, 4, 8, EPI_E3M2, PRO>(a, s);
    } else {
        if (k == 9)
            return go_smallm<M, 6, 2, 4, EPI_E3M2, PRO>(a, s);
        if (k == 10)
            return go_smallm<M, 6, 4, 4, EPI_E3M2, PRO>(a, s);
    }
    return hipErrorInvalidValue;
}

template <int EPI, int PRO>
hipError_t dispatch_rotated(const RotArgs &a, int k, int m, hipStream_t s)
{
    if constexpr (EPI == EPI_E3M2) {
        switch (m) {
        case 1: return k >= 7 ? dispatch_pow2<EPI_E3M2, true, PRO>(a, k, s) : hipErrorInvalidValue;
        case 12: return dispatch_smallm_e3m2<12, PRO>(a, k, s);
        case 20: return dispatch_smallm_e3m2<20, PRO>(a, k, s);
        case 28: return dispatch_smallm_e3m2<28, PRO>(a, k, s);
        case 108:
            return go_largem<108, EPI_E3M2, PRO>(a, s);
        case 172: return go_largem<172, EPI_E3M2, PRO>(a, s);
        }
        return hipErrorInvalidValue;
    } else {
        switch (m) {
        case 1: return dispatch_pow2<EPI, true, PRO>(a, k, s);
        case 12: return dispatch_smallm<12, 8, EPI, PRO>(a, k, s);
        case 20: return dispatch_smallm<20, 4, EPI, PRO>(a, k, s);
        case 28: return dispatch_smallm<28, 4, EPI, PRO>(a, k, s);
        case 108: return go_largem<108, EPI, PRO>(a, s);
        case 172: return go_largem<172, EPI, PRO>(a, s);
        }
    }
    return hipErrorInvalidValue;
}

template <int LOGL, int C>
hipError_t go_kvdeq(const KvDeqArgs &a, bool inv, hipStream_t s)
{
    constexpr int RPB = 4 * (64 >> LOGL);
    const int64_t blocks = (a.rows + RPB - 1) / RPB;
    if (inv)
        hipLaunchKernelGGL((k_kv_dequant<LOGL, C, true>), dim3((unsigned)blocks), dim3(256), 0, s,
                           a);
    else
        hipLaunchKernelGGL((k_kv_dequant<LOGL, C, false>), dim3((unsigned)blocks), dim3(256), 0,
                           s, a);
    return hipGetLastError();
}

}  // namespace


hipError_t launch_rotate(const RotArgs &a, int epi, bool rotate, int k, int m, hipStream_t s,
                         int pro)
{
    if (a.rows == 0)
        return hipSuccess;
    if (pro == PRO_SWIGLU) {
        if (!rotate)
            return hipErrorInvalidValue;
        if (epi == EPI_SYM)
            return dispatch_rotated<EPI_SYM, PRO_SWIGLU>(a, k, m, s);
        if (epi == EPI_E3M2)
            return dispatch_rotated<EPI_E3M2, PRO_SWIGLU>(a, k, m, s);
        return hipErrorInvalidValue;
    }
    if (!rotate) {
        if (epi == EPI_SYM || epi == EPI_SYM8 || epi == EPI_E3M2) {
            if (epi == EPI_SYM)
                hipLaunchKernelGGL(k_quant_plain<EPI_SYM>, dim3((unsigned)a.rows), dim3(256), 0,
                                   s, a);
            else if (epi == EPI_E3M2)
                hipLaunchKernelGGL(k_quant_plain<EPI_E3M2>, dim3((unsigned)a.rows), dim3(256), 0,
                                   s, a);
            else
                hipLaunchKernelGGL(k_quant_plain<EPI_SYM8>, dim3((unsigned)a.rows), dim3(256), 0,
                                   s, a);
            return hipGetLastError();
        }
        if (epi == EPI_KV)
            return a.group == a.n ? dispatch_pow2<EPI_KV, false, PRO_PLAIN, false, true>(a, k, s)
                                  : dispatch_pow2<EPI_KV, false, PRO_PLAIN>(a, k, s);
        return hipErrorInvalidValue;
    }
    if (a.s0 > 0) {  // across heads: n a power of two
        if (m != 1)
            return hipErrorInvalidValue;
        if (epi == EPI_F16)
            return dispatch_pow2<EPI_F16, true, PRO_PLAIN, true>(a, k, s);
        if (epi == EPI_SYM)
            return dispatch_pow2<EPI_SYM, true, PRO_PLAIN, true>(a, k, s);
        return hipErrorInvalidValue;
    }
    switch (epi) {
    case EPI_F32: return dispatch_rotated<EPI_F32, PRO_PLAIN>(a, k, m, s);
    case EPI_F16: return dispatch_rotated<EPI_F16, PRO_PLAIN>(a, k, m, s);
    case EPI_SYM: return dispatch_rotated<EPI_SYM, PRO_PLAIN>(a, k, m, s);
    case EPI_SYM8: return dispatch_rotated<EPI_SYM8, PRO_PLAIN>(a, k, m, s);
    case EPI_E3M2: return dispatch_rotated<EPI_E3M2, PRO_PLAIN>(a, k, m, s);
    case EPI_KV:
        return a.group == a.n ? dispatch_pow2<EPI_KV, true, PRO_PLAIN, false, true>(a, k, s)
                              : dispatch_pow2<EPI_KV, true, PRO_PLAIN>(a, k, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_quant_search(const SearchArgs &a, int bits, bool f32_in, hipStream_t s)
{
    if (a.rows == 0)
        return hipSuccess;
    const dim3 grid((unsigned)a.rows), block(256);
    if (f32_in) {
        if (bits == 4)
            hipLaunchKernelGGL((k_quant_search<4, float>), grid, block, 0, s, a);
        else if (bits == 6)
            hipLaunchKernelGGL((k_quant_search<6, float>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((k_quant_search<8, float>), grid, block, 0, s, a);
    } else {
        if (bits == 4)
            hipLaunchKernelGGL((k_quant_search<4, uint16_t>), grid, block, 0, s, a);
        else if (bits == 6)
            hipLaunchKernelGGL((k_quant_search<6, uint16_t>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((k_quant_search<8, uint16_t>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

template <typename TIN>
static hipError_t quant_grouped_as(const void *y, uint8_t *q, uint16_t *scale, int64_t rows,
                                   int n, int group, float clip, hipStream_t s)
{
    const int logl = ilog2(group / 8);
    const int64_t rpb = 256 >> logl;  // rows per block
    const int64_t blocks = (rows + rpb - 1) / rpb * (n / group);
    if (blocks > 0x7FFFFFFF)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(256);
    switch (logl) {
    case 0: hipLaunchKernelGGL((k_quant_grouped<0, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 1: hipLaunchKernelGGL((k_quant_grouped<1, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 2: hipLaunchKernelGGL((k_quant_grouped<2, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 3: hipLaunchKernelGGL((k_quant_grouped<3, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 4: hipLaunchKernelGGL((k_quant_grouped<4, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 5: hipLaunchKernelGGL((k_quant_grouped<5, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    case 6: hipLaunchKernelGGL((k_quant_grouped<6, TIN>), grid, block, 0, s, y, q, scale, rows, n, clip); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_quant_grouped(const void *y, bool f32_in, uint8_t *q, uint16_t *scale,
                                int64_t rows, int n, int group, float clip, hipStream_t s)
{
    if (group < 8 || group > 512 || (group & (group - 1)) || n % group)
        return hipErrorInvalidValue;
    if (rows == 0)
        return hipSuccess;
    return f32_in ? quant_grouped_as<float>(y, q, scale, rows, n, group, clip, s)
                  : quant_grouped_as<uint16_t>(y, q, scale, rows, n, group, clip, s);
}

hipError_t launch_swiglu(const uint16_t *g, const uint16_t *u, uint16_t *h, int64_t count,
                         hipStream_t s)
{
    const int64_t chunks = count / 8;
    if (chunks == 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((chunks + 255) / 256, 256 * 16);
    hipLaunchKernelGGL(k_swiglu, dim3((unsigned)blocks), dim3(256), 0, s, g, u, h, chunks);
    return hipGetLastError();
}

hipError_t launch_kv_dequant(const KvDeqArgs &a, bool inverse_rotate, hipStream_t s)
{
    if (a.rows == 0)
        return hipSuccess;
    // two chunks (16 elements) per lane: each store instruction then writes
    // 128 contiguous bytes of a row (measured faster than 1 or 4 chunks)
    switch (a.n) {
    case 8: return go_kvdeq<0, 1>(a, inverse_rotate, s);
    case 16: return go_kvdeq<0, 2>(a, inverse_rotate, s);
    case 32: return go_kvdeq<1, 2>(a, inverse_rotate, s);
    case 64: return go_kvdeq<2, 2>(a, inverse_rotate, s);
    case 128: return go_kvdeq<3, 2>(a, inverse_rotate, s);
    case 256: return go_kvdeq<4, 2>(a, inverse_rotate, s);
    case 512: return go_kvdeq<5, 2>(a, inverse_rotate, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace quarot
