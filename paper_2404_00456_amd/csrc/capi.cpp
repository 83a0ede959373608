// C ABI of libquarot: argument validation, size dispatch, launches.
// Every check runs on the host before any device work; on error no output
// is touched.
#include "../../include/quarot.h"

#include <cmath>
#include <cstdlib>
#include <cstring>

#include "common.hpp"
#include "hadamard_factors.hpp"

using namespace quarot;

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kMaxN = 32768;

bool aligned16(const void *p)
{
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// n = 2^k * m with m picked by the odd part of n.
bool factor(int64_t n, int *k, int *m)
{
    if (n <= 0)
        return false;
    static const int ms[6] = {1, 12, 20, 28, 108, 172};
    for (int t = 0; t < 6; ++t) {
        if (n % ms[t])
            continue;
        const int64_t p = n / ms[t];
        if (p & (p - 1))
            continue;
        int kk = 0;
        while ((int64_t(1) << kk) < p)
            ++kk;
        *k = kk;
        *m = ms[t];
        return true;
    }
    return false;
}

// RN32(1/sqrt(n)), through double (exact square root, one division).
float rotation_scale(int64_t n)
{
    return (float)(1.0 / std::sqrt((double)n));
}

bool clip_ok(float c)
{
    return c > 0.0f && c <= 1.0f;
}

quarot_status hip_fail(hipError_t e)
{
    g_last_hip_error = (int)e;
    return QUAROT_ERR_HIP;
}

// Failure injection for tests of the error path: when the environment
// variable QUAROT_FAKE_HIP_ERROR holds the name of an entry point, that
// entry point behaves as if its first HIP runtime call had failed with
// hipErrorLaunchFailure.  It validates its arguments as usual, then returns
// QUAROT_ERR_HIP before any device work (every output untouched), and
// quarot_last_hip_error() reports the code.  Read on every call, so a
// process can set and clear it.
bool fake_hip_error(const char *call)
{
    const char *v = std::getenv("QUAROT_FAKE_HIP_ERROR");
    return v && call && std::strcmp(v, call) == 0;
}

// The device of the calling thread must be a gfx950.  Cached per thread
// and device (a host-side query, no device work).  `call` names the entry
// point (for the failure injection above).
quarot_status check_device(const char *call)
{
    if (fake_hip_error(call))
        return hip_fail(hipErrorLaunchFailure);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return QUAROT_ERR_NO_DEVICE;
    }
    thread_local int ok_dev = -1;
    if (ok_dev == dev)
        return QUAROT_OK;
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return QUAROT_ERR_NO_DEVICE;
    }
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return QUAROT_ERR_NO_DEVICE;
    ok_dev = dev;
    return QUAROT_OK;
}

quarot_status check_rot_size(int64_t n, bool rotate, int epi, int *k, int *m)
{
    if (n <= 0 || n > kMaxN || (n & 7))
        return n <= 0 ? QUAROT_ERR_INVALID_ARG : QUAROT_ERR_UNSUPPORTED_SIZE;
    *k = 0;
    *m = 1;
    if (rotate || epi == EPI_KV) {
        if (!factor(n, k, m))
            return QUAROT_ERR_UNSUPPORTED_SIZE;
    }
    if (!rotate_supported(epi, rotate, *k, *m, (int)n))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    return QUAROT_OK;
}

quarot_status check_gemm_sizes(int64_t M, int64_t N, int64_t K)
{
    if (M < 0 || N < 0 || K <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (K % 64 || K > 65536 || M > (int64_t(1) << 30) || N > (int64_t(1) << 30))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (M > 0 && N > 0 && (int64_t)((M + 255) / 256) * ((N + 255) / 256) > 0x7FFFFFFF)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    return QUAROT_OK;
}

quarot_status check_gemm(const uint8_t *xq, const quarot_f16 *sx, const uint8_t *wq,
                         const quarot_f16 *sw, const quarot_f16 *y, const int32_t *acc,
                         int64_t M, int64_t N, int64_t K)
{
    quarot_status st = check_gemm_sizes(M, N, K);
    if (st || M == 0 || N == 0)
        return st;
    if (!xq || !sx || !wq || !sw || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(xq) || !aligned16(wq) || !aligned16(y) || !aligned16(sx) ||
        !aligned16(sw) || (acc && !aligned16(acc)))
        return QUAROT_ERR_ALIGNMENT;
    return QUAROT_OK;
}

size_t codes_bytes(int64_t M, int64_t K)
{
    return ((size_t)M * (size_t)(K / 2) + 255) & ~(size_t)255;
}

}  // namespace

extern "C" {

const char *quarot_status_string(int status)
{
    switch (status) {
    case QUAROT_OK: return "QUAROT_OK";
    case QUAROT_ERR_INVALID_ARG: return "QUAROT_ERR_INVALID_ARG";
    case QUAROT_ERR_UNSUPPORTED_SIZE: return "QUAROT_ERR_UNSUPPORTED_SIZE";
    case QUAROT_ERR_ALIGNMENT: return "QUAROT_ERR_ALIGNMENT";
    case QUAROT_ERR_WORKSPACE: return "QUAROT_ERR_WORKSPACE";
    case QUAROT_ERR_NO_DEVICE: return "QUAROT_ERR_NO_DEVICE";
    case QUAROT_ERR_HIP: return "QUAROT_ERR_HIP";
    }
    return "QUAROT_ERR_UNKNOWN";
}

int quarot_last_hip_error(void)
{
    return g_last_hip_error;
}

int quarot_version(void)
{
    return 100;  // 0.1.0
}

quarot_status quarot_hadamard_factor(int64_t n, int *log2_pow2, int *m)
{
    if (!log2_pow2 || !m || n <= 0)
        return QUAROT_ERR_INVALID_ARG;
    int k, mm;
    if (n > kMaxN || (n & 7) || !factor(n, &k, &mm) ||
        !rotate_supported(EPI_SYM, true, k, mm, (int)n))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    *log2_pow2 = k;
    *m = mm;
    return QUAROT_OK;
}

quarot_status quarot_hadamard_factor_table(int m, int8_t *out)
{
    if (!out)
        return QUAROT_ERR_INVALID_ARG;
    if (!hm_supported(m))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    for (int r = 0; r < m; ++r)
        for (int s = 0; s < m; ++s)
            out[r * m + s] = (int8_t)hm_sign(m, r, s);
    return QUAROT_OK;
}

quarot_status quarot_hadamard(const quarot_f16 *x, quarot_f16 *y, int64_t rows, int64_t n,
                              void *stream)
{
    if (rows < 0)
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, true, EPI_F16, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!x || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(y))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = x;
    a.out = y;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = 1.0f;
    hipError_t e = launch_rotate(a, EPI_F16, true, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_quant_int4(const quarot_f16 *x, uint8_t *q, quarot_f16 *scale,
                                int64_t rows, int64_t n, int rotate, float clip_ratio,
                                void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, rotate != 0, EPI_SYM, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!x || !q || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(q) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = x;
    a.out = q;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = clip_ratio;
    hipError_t e = launch_rotate(a, EPI_SYM, rotate != 0, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_w4a4_gemm(const uint8_t *xq, const quarot_f16 *sx, const uint8_t *wq,
                               const quarot_f16 *sw, quarot_f16 *y, int32_t *acc_out,
                               int64_t M, int64_t N, int64_t K, void *stream)
{
    quarot_status st = check_gemm(xq, sx, wq, sw, y, acc_out, M, N, K);
    if (st || M == 0 || N == 0)
        return st;
    if ((st = check_device(__func__)))
        return st;
    GemmArgs a{xq, sx, wq, sw, y, acc_out, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm(a, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_pack_e3m2(const uint8_t *q4, uint8_t *q6, int64_t rows, int64_t k,
                               void *stream)
{
    if (rows < 0 || k <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (k % 128 || k > 65536 || rows > (int64_t(1) << 30))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!q4 || !q6)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(q4) || !aligned16(q6))
        return QUAROT_ERR_ALIGNMENT;
    quarot_status st = check_device(__func__);
    if (st)
        return st;
    hipError_t e = launch_pack_e3m2(q4, q6, rows, (int)k, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_w4a4_gemm_e3m2(const uint8_t *xq6, const quarot_f16 *sx,
                                    const uint8_t *wq6, const quarot_f16 *sw, quarot_f16 *y,
                                    int32_t *acc_out, int64_t M, int64_t N, int64_t K,
                                    void *stream)
{
    quarot_status st = check_gemm(xq6, sx, wq6, sw, y, acc_out, M, N, K);
    if (st)
        return st;
    if (K % 128)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (M == 0 || N == 0)
        return QUAROT_OK;
    if ((st = check_device(__func__)))
        return st;
    GemmArgs a{xq6, sx, wq6, sw, y, acc_out, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm(a, (hipStream_t)stream, 6);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_linear_workspace_size(int64_t M, int64_t K)
{
    if (M < 0 || K <= 0 || (K & 1))
        return 0;
    const size_t scales = ((size_t)M * 2 + 255) & ~(size_t)255;
    return codes_bytes(M, K) + scales;
}

quarot_status quarot_linear(const quarot_f16 *x, const uint8_t *wq, const quarot_f16 *sw,
                            quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                            float clip_ratio, void *workspace, size_t workspace_bytes,
                            void *stream)
{
    if (M < 0 || N < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(K, rotate != 0, EPI_SYM, &k, &m);
    if (st)
        return st;
    if ((st = check_gemm_sizes(M, N, K)))
        return st;
    if (M == 0 || N == 0)
        return QUAROT_OK;
    if (!x || !wq || !sw || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(wq) || !aligned16(sw) || !aligned16(y))
        return QUAROT_ERR_ALIGNMENT;
    if (!workspace || workspace_bytes < quarot_linear_workspace_size(M, K))
        return QUAROT_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    uint8_t *xq = static_cast<uint8_t *>(workspace);
    quarot_f16 *sx = reinterpret_cast<quarot_f16 *>(xq + codes_bytes(M, K));
    RotArgs ra{};
    ra.x = x;
    ra.out = xq;
    ra.scale = sx;
    ra.rows = M;
    ra.n = (int)K;
    ra.c = rotation_scale(K);
    ra.clip = clip_ratio;
    hipError_t e = launch_rotate(ra, EPI_SYM, rotate != 0, k, m, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e);
    GemmArgs ga{xq, sx, wq, sw, y, nullptr, (int)M, (int)N, (int)K};
    e = launch_gemm(ga, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_quant_int4_e3m2(const quarot_f16 *x, uint8_t *q6, quarot_f16 *scale,
                                     int64_t rows, int64_t n, int rotate, float clip_ratio,
                                     void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, rotate != 0, EPI_E3M2, &k, &m);
    if (st)
        return st;
    if (rows > (int64_t(1) << 30))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!x || !q6 || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(q6) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = x;
    a.out = q6;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = clip_ratio;
    hipError_t e = launch_rotate(a, EPI_E3M2, rotate != 0, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_linear_e3m2_workspace_size(int64_t M, int64_t K)
{
    if (M < 0 || K <= 0 || (K % 128))
        return 0;
    const size_t codes = ((size_t)M * (size_t)(K / 4 * 3) + 255) & ~(size_t)255;
    const size_t scales = ((size_t)M * 2 + 255) & ~(size_t)255;
    return codes + scales;
}

}  // extern "C"

namespace {

// Checks of the e3m2 layer's arguments other than its workspace; on
// success k, m hold the factorization of K.  *noop is set when there is
// nothing to compute.
quarot_status check_linear_e3m2(const quarot_f16 *x, const uint8_t *wq6, const quarot_f16 *sw,
                                const quarot_f16 *y, int64_t M, int64_t N, int64_t K,
                                int rotate, float clip_ratio, int *k, int *m, bool *noop)
{
    *noop = false;
    if (M < 0 || N < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    quarot_status st = check_rot_size(K, rotate != 0, EPI_E3M2, k, m);
    if (st)
        return st;
    if ((st = check_gemm_sizes(M, N, K)))
        return st;
    if (M == 0 || N == 0) {
        *noop = true;
        return QUAROT_OK;
    }
    if (!x || !wq6 || !sw || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(wq6) || !aligned16(sw) || !aligned16(y))
        return QUAROT_ERR_ALIGNMENT;
    return QUAROT_OK;
}

// The e3m2 layer's two launches with its codes and scales in `workspace`
// (at least quarot_linear_e3m2_workspace_size(M, K) bytes, 256-B aligned).
quarot_status run_linear_e3m2(const quarot_f16 *x, const uint8_t *wq6, const quarot_f16 *sw,
                              quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                              float clip_ratio, int k, int m, void *workspace, void *stream)
{
    uint8_t *xq6 = static_cast<uint8_t *>(workspace);
    const size_t codes = ((size_t)M * (size_t)(K / 4 * 3) + 255) & ~(size_t)255;
    quarot_f16 *sx = reinterpret_cast<quarot_f16 *>(xq6 + codes);
    RotArgs ra{};
    ra.x = x;
    ra.out = xq6;
    ra.scale = sx;
    ra.rows = M;
    ra.n = (int)K;
    ra.c = rotation_scale(K);
    ra.clip = clip_ratio;
    hipError_t e = launch_rotate(ra, EPI_E3M2, rotate != 0, k, m, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e);
    GemmArgs ga{xq6, sx, wq6, sw, y, nullptr, (int)M, (int)N, (int)K};
    e = launch_gemm(ga, (hipStream_t)stream, 6);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

}  // namespace

extern "C" {

quarot_status quarot_linear_e3m2(const quarot_f16 *x, const uint8_t *wq6, const quarot_f16 *sw,
                                 quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                                 float clip_ratio, void *workspace, size_t workspace_bytes,
                                 void *stream)
{
    int k, m;
    bool noop;
    quarot_status st =
        check_linear_e3m2(x, wq6, sw, y, M, N, K, rotate, clip_ratio, &k, &m, &noop);
    if (st || noop)
        return st;
    if (!workspace || workspace_bytes < quarot_linear_e3m2_workspace_size(M, K))
        return QUAROT_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    return run_linear_e3m2(x, wq6, sw, y, M, N, K, rotate, clip_ratio, k, m, workspace, stream);
}

quarot_status quarot_linear_e3m2_scratch(const quarot_f16 *x, const uint8_t *wq6,
                                         const quarot_f16 *sw, quarot_f16 *y, int64_t M,
                                         int64_t N, int64_t K, int rotate, float clip_ratio,
                                         void *stream)
{
    int k, m;
    bool noop;
    quarot_status st =
        check_linear_e3m2(x, wq6, sw, y, M, N, K, rotate, clip_ratio, &k, &m, &noop);
    if (st || noop)
        return st;
    if (quarot_linear_e3m2_workspace_size(M, K) > (size_t)QUAROT_SCRATCH_BYTES)
        return QUAROT_ERR_WORKSPACE;  // beyond the fixed array
    if ((st = check_device(__func__)))
        return st;
    void *ws = nullptr;
    hipError_t e = scratch_buffer(&ws);  // the array's address on this device
    if (e != hipSuccess)
        return hip_fail(e);
    return run_linear_e3m2(x, wq6, sw, y, M, N, K, rotate, clip_ratio, k, m, ws, stream);
}

quarot_status quarot_quant_int8(const quarot_f16 *x, int8_t *q, quarot_f16 *scale, int64_t rows,
                                int64_t n, int rotate, float clip_ratio, int bits, void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio) || (bits != 6 && bits != 8))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, rotate != 0, EPI_SYM8, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!x || !q || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(q) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = x;
    a.out = q;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = clip_ratio;
    a.qmax = (1 << (bits - 1)) - 1;
    hipError_t e = launch_rotate(a, EPI_SYM8, rotate != 0, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_w8a8_gemm(const int8_t *xq, const quarot_f16 *sx, const int8_t *wq,
                               const quarot_f16 *sw, quarot_f16 *y, int32_t *acc_out,
                               int64_t M, int64_t N, int64_t K, void *stream)
{
    const uint8_t *xb = reinterpret_cast<const uint8_t *>(xq);
    const uint8_t *wb = reinterpret_cast<const uint8_t *>(wq);
    quarot_status st = check_gemm(xb, sx, wb, sw, y, acc_out, M, N, K);
    if (st || M == 0 || N == 0)
        return st;
    if ((st = check_device(__func__)))
        return st;
    GemmArgs a{xb, sx, wb, sw, y, acc_out, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm(a, (hipStream_t)stream, 8);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_linear_w8a8_workspace_size(int64_t M, int64_t K)
{
    if (M < 0 || K <= 0)
        return 0;
    const size_t codes = ((size_t)M * (size_t)K + 255) & ~(size_t)255;
    const size_t scales = ((size_t)M * 2 + 255) & ~(size_t)255;
    return codes + scales;
}

quarot_status quarot_linear_w8a8(const quarot_f16 *x, const int8_t *wq, const quarot_f16 *sw,
                                 quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                                 float clip_ratio, int bits, void *workspace,
                                 size_t workspace_bytes, void *stream)
{
    if (M < 0 || N < 0 || !clip_ok(clip_ratio) || (bits != 6 && bits != 8))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(K, rotate != 0, EPI_SYM8, &k, &m);
    if (st)
        return st;
    if ((st = check_gemm_sizes(M, N, K)))
        return st;
    if (M == 0 || N == 0)
        return QUAROT_OK;
    if (!x || !wq || !sw || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(wq) || !aligned16(sw) || !aligned16(y))
        return QUAROT_ERR_ALIGNMENT;
    if (!workspace || workspace_bytes < quarot_linear_w8a8_workspace_size(M, K))
        return QUAROT_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    uint8_t *xq = static_cast<uint8_t *>(workspace);
    quarot_f16 *sx =
        reinterpret_cast<quarot_f16 *>(xq + (((size_t)M * (size_t)K + 255) & ~(size_t)255));
    RotArgs ra{};
    ra.x = x;
    ra.out = xq;
    ra.scale = sx;
    ra.rows = M;
    ra.n = (int)K;
    ra.c = rotation_scale(K);
    ra.clip = clip_ratio;
    ra.qmax = (1 << (bits - 1)) - 1;
    hipError_t e = launch_rotate(ra, EPI_SYM8, rotate != 0, k, m, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e);
    GemmArgs ga{xq, sx, reinterpret_cast<const uint8_t *>(wq), sw, y, nullptr, (int)M, (int)N,
                (int)K};
    e = launch_gemm(ga, (hipStream_t)stream, 8);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_quant_search_workspace_size(int64_t rows, int64_t n, int rotate)
{
    if (rows < 0 || n <= 0 || !rotate)
        return 0;
    return ((size_t)rows * (size_t)n * sizeof(float) + 255) & ~(size_t)255;
}

quarot_status quarot_quant_search(const quarot_f16 *w, void *q, quarot_f16 *scale,
                                  float *clip_out, int64_t rows, int64_t n, int rotate, int bits,
                                  int n_candidates, void *workspace, size_t workspace_bytes,
                                  void *stream)
{
    if (rows < 0 || (bits != 4 && bits != 6 && bits != 8) || n_candidates < 1 ||
        n_candidates > 100)
        return QUAROT_ERR_INVALID_ARG;
    int k, m;  // without rotation the search reads the fp16 rows itself
    quarot_status st = check_rot_size(n, rotate != 0, rotate ? EPI_F32 : EPI_SYM, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!w || !q || !scale || !clip_out)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(w) || !aligned16(q) || !aligned16(scale) || !aligned16(clip_out))
        return QUAROT_ERR_ALIGNMENT;
    const size_t need = quarot_quant_search_workspace_size(rows, n, rotate);
    if (need && (!workspace || workspace_bytes < need))
        return QUAROT_ERR_WORKSPACE;
    if (need && !aligned16(workspace))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    if (rotate) {
        RotArgs a{};
        a.x = w;
        a.out = workspace;
        a.rows = rows;
        a.n = (int)n;
        a.c = rotation_scale(n);
        a.clip = 1.0f;
        hipError_t e = launch_rotate(a, EPI_F32, true, k, m, (hipStream_t)stream);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    SearchArgs sa{};
    sa.y = rotate ? workspace : (const void *)w;
    sa.q = q;
    sa.scale = scale;
    sa.clip = clip_out;
    sa.rows = rows;
    sa.n = (int)n;
    sa.ncand = n_candidates;
    hipError_t e = launch_quant_search(sa, bits, rotate != 0, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

// ---------------------------------------------------------- group-wise ---

namespace {

quarot_status check_group(int64_t n, int64_t group)
{
    if (group <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (group < 8 || group > 512 || (group & (group - 1)) || n % group)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    return QUAROT_OK;
}

quarot_status check_group_quant_grid(int64_t rows, int64_t n, int64_t group)
{
    const int64_t rpb = 256 / (group / 8);  // rows per block of the group quantizer
    if ((rows + rpb - 1) / rpb * (n / group) > 0x7FFFFFFF)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    return QUAROT_OK;
}

quarot_status check_gemm_grouped_sizes(int64_t M, int64_t N, int64_t K, int64_t group)
{
    quarot_status st = check_gemm_sizes(M, N, K);
    if (st)
        return st;
    if (group != 64 && group != 128 && group != 256)
        return group <= 0 ? QUAROT_ERR_INVALID_ARG : QUAROT_ERR_UNSUPPORTED_SIZE;
    if (K % (group < 128 ? 128 : group))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (M > 0 && N > 0 && (int64_t)((M + 255) / 256) * ((N + 127) / 128) > 0x7FFFFFFF)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    return QUAROT_OK;
}

size_t f32_rows_bytes(int64_t rows, int64_t n)
{
    return ((size_t)rows * (size_t)n * sizeof(float) + 255) & ~(size_t)255;
}

// Rotation to binary32 (when asked) and the group quantizer.
quarot_status group_quant(const quarot_f16 *x, uint8_t *q, quarot_f16 *scale, int64_t rows,
                          int64_t n, int64_t group, bool rotate, int k, int m, float clip,
                          void *f32_rows, hipStream_t s)
{
    if (rotate) {
        RotArgs a{};
        a.x = x;
        a.out = f32_rows;
        a.rows = rows;
        a.n = (int)n;
        a.c = rotation_scale(n);
        a.clip = 1.0f;
        hipError_t e = launch_rotate(a, EPI_F32, true, k, m, s);
        if (e != hipSuccess)
            return hip_fail(e);
    }
    hipError_t e = launch_quant_grouped(rotate ? f32_rows : (const void *)x, rotate, q, scale,
                                        rows, (int)n, (int)group, clip, s);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

}  // namespace

size_t quarot_quant_int4_grouped_workspace_size(int64_t rows, int64_t n, int rotate)
{
    if (rows < 0 || n <= 0 || !rotate)
        return 0;
    return f32_rows_bytes(rows, n);
}

quarot_status quarot_quant_int4_grouped(const quarot_f16 *x, uint8_t *q, quarot_f16 *scale,
                                        int64_t rows, int64_t n, int64_t group, int rotate,
                                        float clip_ratio, void *workspace,
                                        size_t workspace_bytes, void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, rotate != 0, rotate ? EPI_F32 : EPI_SYM, &k, &m);
    if (st)
        return st;
    if ((st = check_group(n, group)) || (st = check_group_quant_grid(rows, n, group)))
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!x || !q || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(q) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    const size_t need = quarot_quant_int4_grouped_workspace_size(rows, n, rotate);
    if (need && (!workspace || workspace_bytes < need))
        return QUAROT_ERR_WORKSPACE;
    if (need && !aligned16(workspace))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    return group_quant(x, q, scale, rows, n, group, rotate != 0, k, m, clip_ratio, workspace,
                       (hipStream_t)stream);
}

quarot_status quarot_w4a4_gemm_grouped(const uint8_t *xq, const quarot_f16 *sx,
                                       const uint8_t *wq, const quarot_f16 *sw, quarot_f16 *y,
                                       int64_t M, int64_t N, int64_t K, int64_t group,
                                       void *stream)
{
    quarot_status st = check_gemm_grouped_sizes(M, N, K, group);
    if (st || M == 0 || N == 0)
        return st;
    if ((st = check_gemm(xq, sx, wq, sw, y, nullptr, M, N, K)))
        return st;
    if ((st = check_device(__func__)))
        return st;
    GemmArgs a{xq, sx, wq, sw, y, nullptr, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm_grouped(a, (int)group, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_w4a4_gemm_grouped_e3m2(const uint8_t *xq6, const quarot_f16 *sx,
                                            const uint8_t *wq6, const quarot_f16 *sw,
                                            quarot_f16 *y, int64_t M, int64_t N, int64_t K,
                                            int64_t group, void *stream)
{
    quarot_status st = check_gemm_grouped_sizes(M, N, K, group);
    if (st)
        return st;
    if (group == 64 || M % 8 || N % 8)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (M == 0 || N == 0)
        return QUAROT_OK;
    if ((st = check_gemm(xq6, sx, wq6, sw, y, nullptr, M, N, K)))
        return st;
    if ((st = check_device(__func__)))
        return st;
    GemmArgs a{xq6, sx, wq6, sw, y, nullptr, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm_grouped_e3m2(a, (int)group, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_linear_w4a4_grouped_workspace_size(int64_t M, int64_t K, int64_t group,
                                                 int rotate)
{
    if (M < 0 || K <= 0 || group <= 0 || K % group)
        return 0;
    const size_t scales = ((size_t)(K / group) * (size_t)M * 2 + 255) & ~(size_t)255;
    return codes_bytes(M, K) + scales + (rotate ? f32_rows_bytes(M, K) : 0);
}

quarot_status quarot_linear_w4a4_grouped(const quarot_f16 *x, const uint8_t *wq,
                                         const quarot_f16 *sw, quarot_f16 *y, int64_t M,
                                         int64_t N, int64_t K, int64_t group, int rotate,
                                         float clip_ratio, void *workspace,
                                         size_t workspace_bytes, void *stream)
{
    if (M < 0 || N < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(K, rotate != 0, rotate ? EPI_F32 : EPI_SYM, &k, &m);
    if (st)
        return st;
    if ((st = check_gemm_grouped_sizes(M, N, K, group)) ||
        (st = check_group_quant_grid(M, K, group)))
        return st;
    if (M == 0 || N == 0)
        return QUAROT_OK;
    if (!x || !wq || !sw || !y)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(wq) || !aligned16(sw) || !aligned16(y))
        return QUAROT_ERR_ALIGNMENT;
    if (!workspace ||
        workspace_bytes < quarot_linear_w4a4_grouped_workspace_size(M, K, group, rotate))
        return QUAROT_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    uint8_t *xq = static_cast<uint8_t *>(workspace);
    quarot_f16 *sx = reinterpret_cast<quarot_f16 *>(xq + codes_bytes(M, K));
    void *f32_rows = reinterpret_cast<uint8_t *>(sx) +
                     (((size_t)(K / group) * (size_t)M * 2 + 255) & ~(size_t)255);
    if ((st = group_quant(x, xq, sx, M, K, group, rotate != 0, k, m, clip_ratio, f32_rows,
                          (hipStream_t)stream)))
        return st;
    GemmArgs ga{xq, sx, wq, sw, y, nullptr, (int)M, (int)N, (int)K};
    hipError_t e = launch_gemm_grouped(ga, (int)group, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_swiglu(const quarot_f16 *gate, const quarot_f16 *up, quarot_f16 *h,
                            int64_t count, void *stream)
{
    if (count < 0)
        return QUAROT_ERR_INVALID_ARG;
    if (count % 8)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (count == 0)
        return QUAROT_OK;
    if (!gate || !up || !h)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(gate) || !aligned16(up) || !aligned16(h))
        return QUAROT_ERR_ALIGNMENT;
    quarot_status st = check_device(__func__);
    if (st)
        return st;
    hipError_t e = launch_swiglu(gate, up, h, count, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_swiglu_quant_int4(const quarot_f16 *gate, const quarot_f16 *up, uint8_t *q,
                                       quarot_f16 *scale, int64_t rows, int64_t n,
                                       float clip_ratio, void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, true, EPI_SYM, &k, &m);
    if (st)
        return st;
    if (!rotate_supported(EPI_SYM, true, k, m, (int)n, PRO_SWIGLU))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!gate || !up || !q || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(gate) || !aligned16(up) || !aligned16(q) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = gate;
    a.x2 = up;
    a.out = q;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = clip_ratio;
    hipError_t e = launch_rotate(a, EPI_SYM, true, k, m, (hipStream_t)stream, PRO_SWIGLU);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_swiglu_quant_e3m2(const quarot_f16 *gate, const quarot_f16 *up, uint8_t *q6,
                                       quarot_f16 *scale, int64_t rows, int64_t n,
                                       float clip_ratio, void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio))
        return QUAROT_ERR_INVALID_ARG;
    int k, m;
    quarot_status st = check_rot_size(n, true, EPI_E3M2, &k, &m);
    if (st)
        return st;
    if (!rotate_supported(EPI_E3M2, true, k, m, (int)n, PRO_SWIGLU))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows > (int64_t(1) << 30))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!gate || !up || !q6 || !scale)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(gate) || !aligned16(up) || !aligned16(q6) || !aligned16(scale))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = gate;
    a.x2 = up;
    a.out = q6;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.c = rotation_scale(n);
    a.clip = clip_ratio;
    hipError_t e = launch_rotate(a, EPI_E3M2, true, k, m, (hipStream_t)stream, PRO_SWIGLU);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

}  // extern "C"

namespace {

// Head-wise transform: n = n_heads * head_dim, both powers of two.
quarot_status heads_launch(const char *call, const quarot_f16 *z, void *out,
                           quarot_f16 *scale, int64_t rows, int64_t n_heads,
                           int64_t head_dim, float clip, int epi, void *stream)
{
    if (rows < 0 || n_heads <= 0 || head_dim <= 0 || !clip_ok(clip))
        return QUAROT_ERR_INVALID_ARG;
    if (n_heads < 2 || (n_heads & (n_heads - 1)) || head_dim < 8 ||
        (head_dim & (head_dim - 1)) || n_heads * head_dim > kMaxN)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    const int64_t n = n_heads * head_dim;
    int k = 0, m = 1, s0 = 0;
    while ((int64_t(1) << k) < n)
        ++k;
    while ((int64_t(1) << s0) < head_dim)
        ++s0;
    if (!rotate_supported(epi, true, k, m, (int)n))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!z || !out || (epi == EPI_SYM && !scale))
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(z) || !aligned16(out) || (scale && !aligned16(scale)))
        return QUAROT_ERR_ALIGNMENT;
    quarot_status st = check_device(call);
    if (st)
        return st;
    RotArgs a{};
    a.x = z;
    a.out = out;
    a.scale = scale;
    a.rows = rows;
    a.n = (int)n;
    a.s0 = s0;
    a.c = rotation_scale(n_heads);
    a.clip = clip;
    hipError_t e = launch_rotate(a, epi, true, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

}  // namespace

extern "C" {

quarot_status quarot_hadamard_heads(const quarot_f16 *z, quarot_f16 *y, int64_t rows,
                                    int64_t n_heads, int64_t head_dim, void *stream)
{
    return heads_launch(__func__, z, y, nullptr, rows, n_heads, head_dim, 1.0f, EPI_F16,
                        stream);
}

quarot_status quarot_hadamard_heads_quant_int4(const quarot_f16 *z, uint8_t *q,
                                               quarot_f16 *scale, int64_t rows, int64_t n_heads,
                                               int64_t head_dim, float clip_ratio, void *stream)
{
    return heads_launch(__func__, z, q, scale, rows, n_heads, head_dim, clip_ratio, EPI_SYM,
                        stream);
}

quarot_status quarot_kv_quant(const quarot_f16 *kv, uint8_t *q, quarot_f16 *scale,
                              quarot_f16 *zero, int64_t rows, int64_t head_dim, int64_t group,
                              int rotate, float clip_ratio, void *stream)
{
    if (rows < 0 || !clip_ok(clip_ratio) || head_dim <= 0 || group <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (head_dim < 8 || head_dim > 512 || (head_dim & (head_dim - 1)) || group < 8 ||
        group > head_dim || (group & (group - 1)))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    int k, m;
    quarot_status st = check_rot_size(head_dim, rotate != 0, EPI_KV, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!kv || !q || !scale || !zero)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(kv) || !aligned16(q) || !aligned16(scale) || !aligned16(zero))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = kv;
    a.out = q;
    a.scale = scale;
    a.zero = zero;
    a.rows = rows;
    a.n = (int)head_dim;
    a.group = (int)group;
    a.c = rotation_scale(head_dim);
    a.clip = clip_ratio;
    a.ostride = 1;
    hipError_t e = launch_rotate(a, EPI_KV, rotate != 0, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_kv_append(const quarot_f16 *kv_new, uint8_t *q_cache,
                               quarot_f16 *scale_cache, quarot_f16 *zero_cache, int64_t rows,
                               int64_t s_max, int64_t pos, int64_t head_dim, int64_t group,
                               int rotate, float clip_ratio, void *stream)
{
    if (rows < 0 || s_max <= 0 || pos < 0 || pos >= s_max || !clip_ok(clip_ratio) ||
        head_dim <= 0 || group <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (head_dim < 8 || head_dim > 512 || (head_dim & (head_dim - 1)) || group < 8 ||
        group > head_dim || (group & (group - 1)))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    int k, m;
    quarot_status st = check_rot_size(head_dim, rotate != 0, EPI_KV, &k, &m);
    if (st)
        return st;
    if (rows == 0)
        return QUAROT_OK;
    if (!kv_new || !q_cache || !scale_cache || !zero_cache)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(kv_new) || !aligned16(q_cache) || !aligned16(scale_cache) ||
        !aligned16(zero_cache))
        return QUAROT_ERR_ALIGNMENT;
    if ((st = check_device(__func__)))
        return st;
    RotArgs a{};
    a.x = kv_new;
    a.out = q_cache;
    a.scale = scale_cache;
    a.zero = zero_cache;
    a.rows = rows;
    a.n = (int)head_dim;
    a.group = (int)group;
    a.c = rotation_scale(head_dim);
    a.clip = clip_ratio;
    a.ostride = s_max;
    a.ooff = pos;
    hipError_t e = launch_rotate(a, EPI_KV, rotate != 0, k, m, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

size_t quarot_kv_attention_workspace_size(int64_t nq, int64_t seq_len, int64_t head_dim)
{
    if (nq <= 0 || seq_len <= 0 || head_dim <= 0)
        return 0;
    const int splits = kv_attn_splits(nq, seq_len);
    return splits > 1 ? (size_t)nq * splits * (size_t)(head_dim + 2) * sizeof(float) : 0;
}

quarot_status quarot_kv_decode_attention(const quarot_f16 *q, const uint8_t *k_codes,
                                         const quarot_f16 *k_scale, const quarot_f16 *k_zero,
                                         const uint8_t *v_codes, const quarot_f16 *v_scale,
                                         const quarot_f16 *v_zero, quarot_f16 *out, int64_t nq,
                                         int64_t nkv, int64_t s_max, int64_t seq_len,
                                         int64_t head_dim, int64_t group, float sm_scale,
                                         void *workspace, size_t workspace_bytes, void *stream)
{
    if (nq < 0 || nkv <= 0 || s_max <= 0 || seq_len <= 0 || seq_len > s_max ||
        head_dim <= 0 || group <= 0 || !(sm_scale > 0.0f) || !std::isfinite(sm_scale))
        return QUAROT_ERR_INVALID_ARG;
    if (nq % nkv)
        return QUAROT_ERR_INVALID_ARG;
    if ((head_dim != 64 && head_dim != 128 && head_dim != 256) || group < 32 ||
        group > head_dim || (group & (group - 1)) || s_max > 0x7FFFFFFF || nq > 0x7FFFFFFF)
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (nq == 0)
        return QUAROT_OK;
    if (!q || !k_codes || !k_scale || !k_zero || !v_codes || !v_scale || !v_zero || !out)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k_codes) || !aligned16(k_scale) || !aligned16(k_zero) ||
        !aligned16(v_codes) || !aligned16(v_scale) || !aligned16(v_zero) || !aligned16(out))
        return QUAROT_ERR_ALIGNMENT;
    const size_t need = quarot_kv_attention_workspace_size(nq, seq_len, head_dim);
    if (need && (!workspace || workspace_bytes < need))
        return QUAROT_ERR_WORKSPACE;
    if (need && !aligned16(workspace))
        return QUAROT_ERR_ALIGNMENT;
    quarot_status st = check_device(__func__);
    if (st)
        return st;
    KvAttnArgs a{};
    a.q = q;
    a.kc = k_codes;
    a.ks = k_scale;
    a.kz = k_zero;
    a.vc = v_codes;
    a.vs = v_scale;
    a.vz = v_zero;
    a.out = out;
    a.part = static_cast<float *>(workspace);
    a.nq = nq;
    a.s_max = s_max;
    a.rep = (int)(nq / nkv);
    a.seq_len = (int)seq_len;
    a.D = (int)head_dim;
    a.G = (int)group;
    a.splits = kv_attn_splits(nq, seq_len);
    a.chunk = (int)(((seq_len + a.splits - 1) / a.splits + 63) / 64 * 64);
    a.sm_scale = sm_scale;
    hipError_t e = launch_kv_attention(a, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

quarot_status quarot_kv_dequant(const uint8_t *q, const quarot_f16 *scale,
                                const quarot_f16 *zero, quarot_f16 *out, int64_t rows,
                                int64_t head_dim, int64_t group, int inverse_rotate,
                                void *stream)
{
    if (rows < 0 || head_dim <= 0 || group <= 0)
        return QUAROT_ERR_INVALID_ARG;
    if (head_dim < 8 || head_dim > 512 || (head_dim & (head_dim - 1)) || group < 8 ||
        group > head_dim || (group & (group - 1)))
        return QUAROT_ERR_UNSUPPORTED_SIZE;
    if (rows == 0)
        return QUAROT_OK;
    if (!q || !scale || !zero || !out)
        return QUAROT_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(scale) || !aligned16(zero) || !aligned16(out))
        return QUAROT_ERR_ALIGNMENT;
    quarot_status st = check_device(__func__);
    if (st)
        return st;
    KvDeqArgs a{q, scale, zero, out, rows, (int)head_dim, (int)group,
                rotation_scale(head_dim)};
    hipError_t e = launch_kv_dequant(a, inverse_rotate != 0, (hipStream_t)stream);
    return e == hipSuccess ? QUAROT_OK : hip_fail(e);
}

}  // extern "C"
