// Shared device helpers and internal launch declarations of libquarot.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

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

// One butterfly of the Walsh-Hadamard transform across lanes: lane pairs
// (p, p ^ mask); the lane with the bit clear keeps u_p + u_q, the other
// keeps u_p - u_q (each one rounded op, as in the canonical order).
__device__ __forceinline__ float bfly_lane(float v, int lane, int mask)
{
    float o = __shfl_xor(v, mask);
    return (lane & mask) ? (o - v) : (v + o);
}

}  // namespace quarot
