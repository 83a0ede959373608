/*
 * quarot.h - C ABI of the MI355X (gfx950) QuaRot W4A4 linear-layer hot path.
 *
 * Paper: "QuaRot: Outlier-Free 4-Bit Inference in Rotated LLMs"
 * (Ashkboos et al., arXiv 2404.00456).
 *
 * What the calls compute (row-major everywhere; "RN" is IEEE
 * round-to-nearest-even, "RN16" rounding to binary16):
 *
 *   rotation   y = x . H_n / sqrt(n) for each row, H_n = H_{2^k} (x) H_m
 *              (§3.1 Kronecker construction; §4 Stage 1b online Hadamard),
 *              computed in binary32 (App. A.7) in one fixed order:
 *              the m-factor sum left to right, then the Walsh-Hadamard
 *              butterflies bit 0 first, then one multiply by RN32(1/sqrt(n)).
 *   quantize   per row (token) symmetric int4 (§4 Stage 2b):
 *              s = RN16(RN(RN(absmax * clip) / 7)),
 *              q = clamp(rint_even(RN(y / s)), -8, 7).
 *   GEMM       acc[m][n] = sum_k qx[m][k] * qw[n][k] in int32
 *              (App. A.10: int4 x int4 -> int32).
 *   dequant    Y[m][n] = RN16(RN(RN(float(acc) * sx[m]) * sw[n]))
 *              (§4 Stage 2b: row scale times column scale).
 *   KV cache   per group of `group` values of a head row, asymmetric
 *              uint4 with clip (§5 Setup: group 128, clip 0.95).
 *
 * Packed int4 layout: byte j of a row holds element 2j in its low nibble
 * and element 2j+1 in its high nibble (two's complement for the signed
 * codes, plain 0..15 for the KV codes).  fp16 values travel as their
 * IEEE binary16 bit patterns (quarot_f16).
 *
 * Conventions for every call:
 *  - Pointers are device pointers (hipMalloc or torch CUDA tensors) unless
 *    stated otherwise, and must be 16-byte aligned.  The caller owns every
 *    buffer, including the workspace; the library never allocates, frees
 *    or keeps pointers, holds no mutable global state and is reentrant.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    Calls only enqueue work on `stream` and return without synchronizing.
 *  - Invalid arguments are reported before any device work, leaving every
 *    output untouched.  A failed launch returns QUAROT_ERR_HIP, and the raw
 *    hipError_t is available from quarot_last_hip_error() on that thread.
 *    Faults inside a kernel surface at the caller's next synchronization.
 *  - Inputs must be finite; results for inf/nan inputs are unspecified.
 */
#ifndef QUAROT_H
#define QUAROT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t quarot_f16; /* IEEE binary16 bits */

typedef enum {
    QUAROT_OK = 0,
    QUAROT_ERR_INVALID_ARG = 1,     /* null pointer, non-positive size, bad clip, ... */
    QUAROT_ERR_UNSUPPORTED_SIZE = 2, /* n has no 2^k * m factorization / kernel */
    QUAROT_ERR_ALIGNMENT = 3,       /* a pointer is not 16-byte aligned */
    QUAROT_ERR_WORKSPACE = 4,       /* workspace missing or too small */
    QUAROT_ERR_NO_DEVICE = 5,       /* no usable gfx950 device */
    QUAROT_ERR_HIP = 6              /* a HIP runtime call failed */
} quarot_status;

/* Human-readable name of a status code (static string, never NULL). */
const char *quarot_status_string(int status);

/* Raw hipError_t of the last QUAROT_ERR_HIP on the calling thread (0 if none). */
int quarot_last_hip_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int quarot_version(void);

/*
 * Which n the rotation supports (§3.1: n = 2^k * m with H_m a known
 * Hadamard matrix).  On success writes k and m.  Host-only, no device use.
 * Supported m: 1 (Sylvester), 12, 20, 108 (Paley I, q = 11, 19, 107),
 * 28 (Paley II, q = 13), 172 (Goethals-Seidel, order-6 cyclotomy of Z_43);
 * n must also be a multiple of 8 and at most 32768.
 * Returns QUAROT_OK, QUAROT_ERR_INVALID_ARG or QUAROT_ERR_UNSUPPORTED_SIZE.
 */
quarot_status quarot_hadamard_factor(int64_t n, int *log2_pow2, int *m);

/*
 * The +-1 factor H_m the library compiles in, row-major into the HOST
 * buffer out[m*m] (entry (r, s) at out[r*m + s]), so that callers can
 * reproduce H_n = H_{2^k} (x) H_m exactly.  Host-only.
 */
quarot_status quarot_hadamard_factor_table(int m, int8_t *out);

/*
 * Standalone online Hadamard (§4 Stage 1b): y[rows][n] = RN16(rotation of x).
 * x, y: fp16 [rows, n]; x == y (in place) is allowed, other overlap is not.
 * rows >= 0 (0 is a no-op), n supported by quarot_hadamard_factor.
 */
quarot_status quarot_hadamard(const quarot_f16 *x, quarot_f16 *y, int64_t rows, int64_t n,
                              void *stream);

/*
 * Per-token symmetric int4 quantization (§4 Stage 2b), optionally of the
 * rotated row (rotate != 0: the binary32 rotation is quantized directly,
 * without an fp16 round trip).
 *   x     fp16 [rows, n]           q     uint8 [rows, n/2] packed codes
 *   scale fp16 [rows] (s above)    clip_ratio in (0, 1] (paper: 0.9; 1 = none)
 * rotate != 0 needs n supported by quarot_hadamard_factor; rotate == 0 needs
 * n a positive multiple of 8.  Also used offline for the weights: each
 * output-channel row of W [N, K] rotated like an activation row and
 * quantized per row gives the per-output-channel wq and sw below
 * (x W^T = (x H)(W H)^T / n, §3.4 computational invariance).
 */
quarot_status quarot_quant_int4(const quarot_f16 *x, uint8_t *q, quarot_f16 *scale,
                                int64_t rows, int64_t n, int rotate, float clip_ratio,
                                void *stream);

/*
 * W4A4 GEMM with fused dequant (§4 Stage 2b, App. A.10):
 *   xq uint8 [M, K/2], sx fp16 [M]     (activations, per-token scales)
 *   wq uint8 [N, K/2], sw fp16 [N]     (weights, per-output-channel scales)
 *   y  fp16 [M, N] = RN16(RN(RN(float(acc) * sx[m]) * sw[n]))
 *   acc_out int32 [M, N] or NULL: the exact integer accumulators.
 * M, N >= 0 (0 is a no-op); K a positive multiple of 64, at most 65536.
 */
quarot_status quarot_w4a4_gemm(const uint8_t *xq, const quarot_f16 *sx, const uint8_t *wq,
                               const quarot_f16 *sw, quarot_f16 *y, int32_t *acc_out,
                               int64_t M, int64_t N, int64_t K, void *stream);

/*
 * Bytes of device workspace quarot_linear needs for M rows of width K:
 * the packed codes (M*K/2) and scales (2*M), each rounded up to 256 bytes.
 * Host-only; returns 0 for invalid sizes.
 */
size_t quarot_linear_workspace_size(int64_t M, int64_t K);

/*
 * The whole 4-bit linear layer (App. A.10): quarot_quant_int4(x, rotate,
 * clip_ratio) into the workspace, then quarot_w4a4_gemm into y.  Two
 * launches on `stream`, nothing else.
 *   x fp16 [M, K], wq uint8 [N, K/2], sw fp16 [N], y fp16 [M, N],
 *   workspace: device memory of at least quarot_linear_workspace_size(M, K)
 *   bytes, 256-byte aligned, not overlapping any other argument.
 * K must satisfy both calls' size rules.
 */
quarot_status quarot_linear(const quarot_f16 *x, const uint8_t *wq, const quarot_f16 *sw,
                            quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                            float clip_ratio, void *workspace, size_t workspace_bytes,
                            void *stream);

/*
 * 4-bit KV cache quantization (§4 Stage 1d: head-wise rotation of keys,
 * and of values via the fused W_v/W_out Hadamard; §5 Setup: asymmetric,
 * group 128, clip 0.95).  rows = batch * heads * tokens vectors of head_dim:
 *   kv fp16 [rows, head_dim]   q uint8 [rows, head_dim/2] (codes 0..15)
 *   scale, zero fp16 [rows, head_dim/group]
 * Per group: mx = RN(max * clip), mn = RN(min * clip),
 *   scale = RN16(RN(RN(mx - mn) / 15)), zero = RN16(mn),
 *   q = clamp(rint_even(RN(RN(y - zero) / scale)), 0, 15); scale 0 -> q 0.
 * rotate != 0 applies H_head_dim / sqrt(head_dim) to each row first.
 * head_dim a power of two in [8, 512]; group a power of two with
 * 8 <= group <= head_dim.
 */
quarot_status quarot_kv_quant(const quarot_f16 *kv, uint8_t *q, quarot_f16 *scale,
                              quarot_f16 *zero, int64_t rows, int64_t head_dim, int64_t group,
                              int rotate, float clip_ratio, void *stream);

/*
 * Dequantize the 4-bit KV cache: out = RN16(yhat) with
 * yhat = RN(RN(float(q) * scale) + zero) (the rotated basis), or, with
 * inverse_rotate != 0, the binary32 rotation of yhat by H_head_dim/sqrt
 * (the Sylvester rotation is its own inverse) before the RN16.
 * Layouts and size rules as quarot_kv_quant.
 */
quarot_status quarot_kv_dequant(const uint8_t *q, const quarot_f16 *scale,
                                const quarot_f16 *zero, quarot_f16 *out, int64_t rows,
                                int64_t head_dim, int64_t group, int inverse_rotate,
                                void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QUAROT_H */
