// Measurement utilities (not steps of the method): MFMA-only loops that give
// the attainable rate of v_mfma_i32_16x16x64_i8 (the int4-operand GEMM's
// instruction) and of v_mfma_f32_16x16x128_f8f6f4 on e3m2 operands (the
// e3m2-operand GEMM's) under load, against which the GEMMs' achieved rates
// can be read besides the published peaks.
//
// Each block is 512 threads (8 waves, two per SIMD, as the GEMM runs); a
// wave keeps 8 independent accumulators and cycles through 4 operand pairs
// drawn from a per-lane hash, so the multipliers see changing data.  Each
// thread writes one int32 (the accumulator sum) so nothing is dead code.
#include "common.hpp"

namespace quarot {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(512, 1) void k_mfma_probe(int32_t *out, int iters)
{
    v4i a[4], b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const unsigned h = (threadIdx.x + 977u * u + 131u * blockIdx.x) * 2654435761u;
        a[u] = v4i{(int)h, (int)(h * 3u), (int)(h ^ 0x5A5A5A5Au), (int)(h * 7u)};
        b[u] = v4i{(int)(h * 11u), (int)(h ^ 0xA5A5A5A5u), (int)(h * 13u), (int)(h + 12345u)};
    }
    v4i acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        acc[i] = v4i{0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[u], b[(u + i) & 3], acc[i], 0,
                                                               0, 0);
    }
    int s = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
    out[(int64_t)blockIdx.x * 512 + threadIdx.x] = s;
}

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

// Same shape with e3m2 operands (six dwords used of eight; any 6-bit field
// is a finite e3m2 number of magnitude <= 28).
__global__ __launch_bounds__(512, 1) void k_mfma_probe_fp6(int32_t *out, int iters)
{
    v8i a[4], b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const unsigned h = (threadIdx.x + 977u * u + 131u * blockIdx.x) * 2654435761u;
#pragma unroll
        for (int d = 0; d < 8; ++d) {
            a[u][d] = d < 6 ? (int)(h * (2u * d + 3u) + d * 0x9E3779B9u) : 0;
            b[u][d] = d < 6 ? (int)((h ^ 0xA5A5A5A5u) * (2u * d + 5u) + d * 0x7F4A7C15u) : 0;
        }
    }
    v4f acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        acc[i] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
                    a[u], b[(u + i) & 3], acc[i], 3, 3, 0, 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
    out[(int64_t)blockIdx.x * 512 + threadIdx.x] = __float_as_int(s);
}

}  // namespace

hipError_t launch_mfma_probe_fp6(int32_t *out, int blocks, int iters, hipStream_t s)
{
    hipLaunchKernelGGL(k_mfma_probe_fp6, dim3((unsigned)blocks), dim3(512), 0, s, out, iters);
    return hipGetLastError();
}

hipError_t launch_mfma_probe(int32_t *out, int blocks, int iters, hipStream_t s)
{
    hipLaunchKernelGGL(k_mfma_probe, dim3((unsigned)blocks), dim3(512), 0, s, out, iters);
    return hipGetLastError();
}

}  // namespace quarot
