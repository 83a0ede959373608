// Drives the C ABI's host code with no device: argument validation of every
// entry point (null, negative, oversized and misaligned arguments, extreme
// sizes), the no-device path of valid calls, the failure injection of
// QUAROT_FAKE_HIP_ERROR and the workspace size queries.  Built with the
// address and undefined-behaviour sanitizers by tests/test_sanitizers.py
// against counting stand-ins of the kernel launchers; fake pointers are
// never dereferenced because nothing launches.
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "quarot.h"

static int failures = 0;
extern int quarot_stub_launches;  // tests/native/launch_stubs.cpp

#define EXPECT(call, want)                                                                   \
    do {                                                                                     \
        const int got_ = (int)(call);                                                        \
        if (got_ != (int)(want)) {                                                           \
            std::printf("FAIL line %d: %s -> %d, want %d\n", __LINE__, #call, got_, (int)(want)); \
            ++failures;                                                                      \
        }                                                                                    \
    } while (0)

int main()
{
    void *P = reinterpret_cast<void *>(uintptr_t(1) << 20);
    void *P2 = reinterpret_cast<void *>((uintptr_t(1) << 20) + 4096);
    void *U = reinterpret_cast<void *>((uintptr_t(1) << 20) + 8);
    const quarot_f16 *H = static_cast<const quarot_f16 *>(P);
    quarot_f16 *H2 = static_cast<quarot_f16 *>(P2);
    uint8_t *B = static_cast<uint8_t *>(P2);
    const int64_t BIG = INT64_C(1) << 62;

    // host-only queries
    int k = -1, m = -1;
    EXPECT(quarot_hadamard_factor(11008, &k, &m), QUAROT_OK);
    EXPECT(k * 1000 + m, 6172);
    EXPECT(quarot_hadamard_factor(BIG, &k, &m), QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_hadamard_factor(-8, &k, &m), QUAROT_ERR_INVALID_ARG);
    int8_t tab[172 * 172];
    EXPECT(quarot_hadamard_factor_table(172, tab), QUAROT_OK);
    EXPECT(quarot_hadamard_factor_table(7, tab), QUAROT_ERR_UNSUPPORTED_SIZE);
    for (int s = -2; s < 9; ++s)
        if (!quarot_status_string(s))
            ++failures;
    EXPECT(quarot_linear_workspace_size(BIG, 8192) == 0 ||
               quarot_linear_workspace_size(BIG, 8192) > 0, 1);
    EXPECT(quarot_linear_e3m2_workspace_size(3, 192), 0);
    EXPECT(quarot_linear_e3m2_workspace_size(-1, 256), 0);
    EXPECT(quarot_kv_attention_workspace_size(BIG, BIG, 128) >= 0, 1);
    EXPECT(quarot_quant_search_workspace_size(BIG, BIG, 1) >= 0, 1);
    EXPECT(quarot_linear_w4a4_grouped_workspace_size(BIG, BIG, 128, 1) >= 0, 1);

    // invalid arguments, before any device query
    EXPECT(quarot_hadamard(nullptr, H2, 4, 128, nullptr), QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_hadamard(H, H2, -1, 128, nullptr), QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_hadamard(H, H2, BIG, 128, nullptr) != QUAROT_OK, 1);
    EXPECT(quarot_hadamard(static_cast<const quarot_f16 *>(U), H2, 4, 128, nullptr),
           QUAROT_ERR_ALIGNMENT);
    EXPECT(quarot_quant_int4(H, B, H2, 4, 128, 1, 0.0f, nullptr), QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_quant_int4(H, B, H2, 4, 100, 1, 1.0f, nullptr), QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_w4a4_gemm(B, H, B, H, H2, nullptr, 4, 4, 100, nullptr),
           QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_w4a4_gemm(B, H, B, H, H2, nullptr, BIG, BIG, 128, nullptr),
           QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_w4a4_gemm_e3m2(B, H, B, H, H2, nullptr, 4, 4, 192, nullptr),
           QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_linear(H, B, H, H2, 4, 4, 128, 1, 1.0f, P, 16, nullptr), QUAROT_ERR_WORKSPACE);
    EXPECT(quarot_linear_e3m2(H, B, H, H2, 4, 4, 128, 1, 1.0f, nullptr, 1 << 20, nullptr),
           QUAROT_ERR_WORKSPACE);
    EXPECT(quarot_linear_e3m2_scratch(H, B, H, H2, 16384, 4, 8192, 1, 1.0f, nullptr),
           QUAROT_ERR_WORKSPACE);
    EXPECT(quarot_linear_e3m2_scratch(H, B, H, H2, BIG, 4, 8192, 1, 1.0f, nullptr) != QUAROT_OK, 1);
    EXPECT(quarot_quant_int8(H, static_cast<int8_t *>(P2), H2, 4, 128, 1, 1.0f, 7, nullptr),
           QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_quant_search(H, P2, H2, static_cast<float *>(P2), 4, 128, 1, 4, 101, P,
                               1 << 20, nullptr),
           QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_quant_int4_grouped(H, B, H2, 4, 256, 96, 1, 1.0f, P, 1 << 20, nullptr) != 0, 1);
    EXPECT(quarot_w4a4_gemm_grouped(B, H, B, H, H2, 4, 4, 256, 32, nullptr) != 0, 1);
    EXPECT(quarot_w4a4_gemm_grouped_e3m2(B, H, B, H, H2, 8, 8, 256, 64, nullptr) != 0, 1);
    EXPECT(quarot_w4a4_gemm_grouped_e3m2(B, H, B, H, H2, 12, 8, 256, 128, nullptr) != 0, 1);
    EXPECT(quarot_kv_quant(H, B, H2, H2, 4, 128, 256, 1, 0.95f, nullptr),
           QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_kv_dequant(B, H, H, H2, 4, 96, 32, 0, nullptr) != 0, 1);
    EXPECT(quarot_kv_append(H, B, H2, H2, 4, 10, 10, 128, 128, 1, 0.95f, nullptr) != 0, 1);
    EXPECT(quarot_kv_decode_attention(H, B, H, H, B, H, H, H2, 4, 3, 64, 64, 128, 128, 0.1f,
                                      P, 1 << 20, nullptr) != 0, 1);
    EXPECT(quarot_hadamard_heads(H, H2, 4, 3, 128, nullptr), QUAROT_ERR_UNSUPPORTED_SIZE);
    EXPECT(quarot_swiglu(H, H, H2, 7, nullptr) != 0, 1);

    // valid calls with no device stop at the device check
    EXPECT(quarot_hadamard(H, H2, 4, 11008, nullptr), QUAROT_ERR_NO_DEVICE);
    EXPECT(quarot_quant_int4_e3m2(H, B, H2, 4, 11008, 1, 1.0f, nullptr), QUAROT_ERR_NO_DEVICE);
    EXPECT(quarot_linear_e3m2_scratch(H, B, H, H2, 2048, 4, 28672, 1, 1.0f, nullptr),
           QUAROT_ERR_NO_DEVICE);
    EXPECT(quarot_kv_quant(H, B, H2, H2, 4, 128, 128, 1, 0.95f, nullptr), QUAROT_ERR_NO_DEVICE);

    // the failure injection comes after validation and before the device
    setenv("QUAROT_FAKE_HIP_ERROR", "quarot_linear", 1);
    EXPECT(quarot_linear(H, B, H, H2, 4, 4, 128, 1, 1.0f, P, 1 << 20, nullptr), QUAROT_ERR_HIP);
    EXPECT(quarot_last_hip_error(), 719);
    EXPECT(quarot_linear(H, B, H, H2, 4, 4, 128, 1, 0.0f, P, 1 << 20, nullptr),
           QUAROT_ERR_INVALID_ARG);
    EXPECT(quarot_hadamard(H, H2, 4, 128, nullptr), QUAROT_ERR_NO_DEVICE);
    unsetenv("QUAROT_FAKE_HIP_ERROR");
    EXPECT(quarot_linear(H, B, H, H2, 4, 4, 128, 1, 1.0f, P, 1 << 20, nullptr),
           QUAROT_ERR_NO_DEVICE);

    EXPECT(quarot_stub_launches, 0);  // nothing tried to launch
    if (failures) {
        std::printf("%d failure(s)\n", failures);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
