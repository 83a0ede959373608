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
};

struct RotArgs {
    const uint16_t *x;  // fp16 [rows, n]
    void *out;          // EPI_F16: fp16 [rows, n]; else uint8 codes [rows, n/2]
    uint16_t *scale;    // EPI_SYM: [rows]; EPI_KV: [rows, n/group]
    uint16_t *zero;     // EPI_KV: [rows, n/group]
    int64_t rows;
    int n;
    int group;          // EPI_KV group size
    float c;            // RN32(1/sqrt(n))
    float clip;
};

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
hipError_t launch_rotate(const RotArgs &a, int epi, bool rotate, int k, int m, hipStream_t s);
hipError_t launch_gemm(const GemmArgs &a, hipStream_t s);
hipError_t launch_kv_dequant(const KvDeqArgs &a, bool inverse_rotate, hipStream_t s);

// Is (k, m) covered by a compiled rotate kernel for this epilogue?
bool rotate_supported(int epi, bool rotate, int k, int m, int n);

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

// One Walsh-Hadamard butterfly across lane bit J: lanes with the bit clear
// get RN(u_lo + u_hi), lanes with it set RN(u_lo - u_hi), each exactly one
// rounded operation as in the canonical order: fma(x, +-1, y) = RN(y +- x).
// s is +1 on lanes with bit J clear and -1 where it is set.
template <int J>
__device__ __forceinline__ float bfly_lane(float v, float s)
{
    if constexpr (J <= 3) {
        return __builtin_fmaf(v, s, lane_xor_dpp<J>(v));  // v is u_lo (s=+1) or u_hi (s=-1)
    } else {
        const float2 p = lane_pair_swap<J>(v);
        return __builtin_fmaf(p.y, s, p.x);
    }
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

// Compile-time loop helper: f(std::integral_constant<int, J>) for J < N.
template <int N, int J = 0, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (J < N) {
        f(std::integral_constant<int, J>());
        static_for<N, J + 1>(f);
    }
}

// Lane signs for the butterflies: +1 where lane bit J is clear, -1 where set.
__device__ __forceinline__ float lane_sign(int lane, int J)
{
    return ((lane >> J) & 1) ? -1.0f : 1.0f;
}

}  // namespace quarot
