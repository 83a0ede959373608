// libquarot_probe (include/quarot_probe.h), built apart from libquarot.
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
#include "../../include/quarot_probe.h"

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

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

thread_local int g_probe_hip_error = 0;

quarot_status hip_fail(hipError_t e)
{
    g_probe_hip_error = (int)e;
    return QUAROT_ERR_HIP;
}

// the current device is a gfx950
quarot_status check_device()
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        g_probe_hip_error = (int)e;
        return QUAROT_ERR_NO_DEVICE;
    }
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
        g_probe_hip_error = (int)e;
        return QUAROT_ERR_NO_DEVICE;
    }
    return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? QUAROT_OK : QUAROT_ERR_NO_DEVICE;
}

quarot_status check_probe(const int32_t *out, int64_t blocks, int iters)
{
    if (blocks <= 0 || blocks > (1 << 20) || iters <= 0 || iters > (1 << 20) || !out)
        return QUAROT_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(out) & 15u)
        return QUAROT_ERR_ALIGNMENT;
    return check_device();
}

}  // namespace

extern "C" {

quarot_status quarot_device_peaks(int *cu_count, int *max_clock_khz)
{
    if (!cu_count || !max_clock_khz)
        return QUAROT_ERR_INVALID_ARG;
    quarot_status st = check_device();
    if (st)
        return st;
    int dev = 0, cus = 0, clk = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&clk, hipDeviceAttributeClockRate, dev);
    if (e != hipSuccess)
        return hip_fail(e);
    *cu_count = cus;
    *max_clock_khz = clk;
    return QUAROT_OK;
}

quarot_status quarot_mfma_probe(int32_t *out, int64_t blocks, int iters, void *stream)
{
    quarot_status st = check_probe(out, blocks, iters);
    if (st)
        return st;
    hipLaunchKernelGGL(k_mfma_probe, dim3((unsigned)blocks), dim3(512), 0, (hipStream_t)stream,
                       out, iters);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_mfma_probe_fp6(int32_t *out, int64_t blocks, int iters, void *stream)
{
    quarot_status st = check_probe(out, blocks, iters);
    if (st)
        return st;
    hipLaunchKernelGGL(k_mfma_probe_fp6, dim3((unsigned)blocks), dim3(512), 0,
                       (hipStream_t)stream, out, iters);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

int quarot_probe_last_hip_error(void)
{
    return g_probe_hip_error;
}

}  // extern "C"
