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
 *              computed in binary32 (App. A.7): element i = a*m + b; the
 *              m-factor sum over b taken exactly and rounded once to
 *              binary32; then the Walsh-Hadamard butterflies over a, bit 0
 *              first, each output one rounded add or subtract; then one
 *              multiply by RN32(1/sqrt(n)); a zero output is +0.
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
 *    or keeps pointers, and is reentrant.  Its one piece of mutable global
 *    state is the fixed scratch array of quarot_linear_e3m2_scratch (see
 *    there); every other call uses only its arguments.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    Calls only enqueue work on `stream` and return without synchronizing.
 *  - Invalid arguments are reported before any device work, leaving every
 *    output untouched.  A failed launch returns QUAROT_ERR_HIP, and the raw
 *    hipError_t is available from quarot_last_hip_error() on that thread.
 *    Faults inside a kernel surface at the caller's next synchronization.
 *  - Inputs must be finite; results for inf/nan inputs are unspecified.
 *  - Failure injection (for tests of callers' error paths): while the
 *    environment variable QUAROT_FAKE_HIP_ERROR holds the name of an entry
 *    point (e.g. "quarot_linear"), that entry point validates its arguments
 *    as usual and then returns QUAROT_ERR_HIP as if its first HIP runtime
 *    call had failed with hipErrorLaunchFailure, before any device work;
 *    quarot_last_hip_error() then returns that code.  The variable is read
 *    on every call.
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

/* Human-readable name of a status code (static string, never NULL).  Takes
 * an int rather than quarot_status so that any integer, also one that is no
 * status, is a valid argument ("QUAROT_ERR_UNKNOWN"). */
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
 * int4 codes in the tiled e3m2 operand layout.  gfx950 has no int4 matrix
 * instruction; its fp6 one (v_mfma_f32_16x16x128_f8f6f4) takes 128-deep
 * slices at twice the int8 rate.  Every code q in -8..8 is exact as an e3m2
 * number (sign, 3 exponent bits of bias 3, 2 mantissa bits), so the
 * products and the binary32 sums of them (integers below 2^24 for
 * K <= 65536) are the exact integer dot products of §4 Stage 2b.
 * Layout of a [rows, K] code matrix, 6 bits per code (1.5 times the int4
 * bytes): K/128 blocks of rows * 96 bytes.  In block b, unit u = 0..3 of
 * row r holds the codes of k = 128 b + 32 u + e (e = 0..31) as the 192-bit
 * word sum_e e3m2(q_e) << 6e.  Its dwords 0-3 (the head) sit at byte
 * r * 64 + 16 (u ^ ((r >> 1) & 3)) of the block; its dwords 4-5 (the tail)
 * at byte rows * 64 + r * 32 + 8 (u ^ ((r >> 2) & 3)).  A 256-row tile's
 * k-block is then two runs of consecutive bytes, and the slot swizzles
 * spread the GEMM's LDS reads over all banks.
 *
 * quarot_pack_e3m2: q4 uint8 [rows, k/2] int4 codes (low nibble first, as
 * quarot_quant_int4 writes them) -> q6 (rows * k * 3/4 bytes, layout above).
 * rows >= 0 (0 is a no-op); k a positive multiple of 128, at most 65536;
 * q4 and q6 16-byte aligned and not overlapping.  Meant for the weights,
 * once per matrix.
 */
quarot_status quarot_pack_e3m2(const uint8_t *q4, uint8_t *q6, int64_t rows, int64_t k,
                               void *stream);

/*
 * quarot_w4a4_gemm with both operands in the tiled e3m2 layout: the same y
 * and acc_out, bit for bit.
 *   xq6 M * K * 3/4 bytes, sx fp16 [M]
 *   wq6 N * K * 3/4 bytes, sw fp16 [N]
 * M, N >= 0 (0 is a no-op); K a positive multiple of 128, at most 65536.
 */
quarot_status quarot_w4a4_gemm_e3m2(const uint8_t *xq6, const quarot_f16 *sx,
                                    const uint8_t *wq6, const quarot_f16 *sw, quarot_f16 *y,
                                    int32_t *acc_out, int64_t M, int64_t N, int64_t K,
                                    void *stream);

/*
 * quarot_quant_int4 with the codes written in the tiled e3m2 layout above:
 * the same codes and scales (§4 Stage 2b), for quarot_w4a4_gemm_e3m2.
 *   x fp16 [rows, n], q6 rows * n * 3/4 bytes, scale fp16 [rows]
 * n a multiple of 128 and, with rotate != 0, n = 2^k (k <= 15) or
 * n = 12 * 2^10, 12 * 2^11, 20 * 2^9, 20 * 2^10, 28 * 2^9, 28 * 2^10,
 * 108 * 2^k (5 <= k <= 7), 172 * 2^k (k = 5, 6); rows <= 2^30.  Other n:
 * quarot_quant_int4 then quarot_pack_e3m2.
 */
quarot_status quarot_quant_int4_e3m2(const quarot_f16 *x, uint8_t *q6, quarot_f16 *scale,
                                     int64_t rows, int64_t n, int rotate, float clip_ratio,
                                     void *stream);

/*
 * The 4-bit linear layer on the e3m2 path: quarot_quant_int4_e3m2 of x into
 * the workspace, then quarot_w4a4_gemm_e3m2 into y (two launches).  The
 * weights come from quarot_quant_int4 of W [N, K] then quarot_pack_e3m2.
 * y equals quarot_linear's bit for bit.  Workspace: at least
 * quarot_linear_e3m2_workspace_size(M, K) bytes, 256-byte aligned (0 for
 * invalid sizes).  Size rules of both calls apply.
 */
size_t quarot_linear_e3m2_workspace_size(int64_t M, int64_t K);
quarot_status quarot_linear_e3m2(const quarot_f16 *x, const uint8_t *wq6, const quarot_f16 *sw,
                                 quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                                 float clip_ratio, void *workspace, size_t workspace_bytes,
                                 void *stream);

/*
 * quarot_linear_e3m2 for callers that cannot allocate device memory (code
 * under HIP graph capture, allocation-free serving loops, harnesses that
 * forbid hipMalloc): the same two launches and the same y bit for bit, with
 * the activation codes and scales in a fixed device array inside the
 * library instead of a workspace.  The array holds QUAROT_SCRATCH_BYTES on
 * every device the library runs on, until the process ends; sizes with
 * quarot_linear_e3m2_workspace_size(M, K) > QUAROT_SCRATCH_BYTES return
 * QUAROT_ERR_WORKSPACE before any device work (e.g. M = 2048 tokens at
 * K = 28672 fit; M = 16384 at K = 8192 does not).  Nothing is allocated; the
 * first call on a device looks up the array's address there
 * (hipGetSymbolAddress), so make one call before capturing a graph.  All
 * calls on one device share the array and it keeps the last call's
 * contents (each call writes all it reads, nothing needs to start at
 * zero): calls that overlap in time on one device, from other streams or
 * threads, race, and the caller must order them.  Other size, pointer and
 * error rules as quarot_linear_e3m2.
 */
#define QUAROT_SCRATCH_BYTES (64u << 20)
quarot_status quarot_linear_e3m2_scratch(const quarot_f16 *x, const uint8_t *wq6,
                                         const quarot_f16 *sw, quarot_f16 *y, int64_t M,
                                         int64_t N, int64_t K, int rotate, float clip_ratio,
                                         void *stream);

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
 * 6- and 8-bit variants of the same scheme (§5.3 round-to-nearest ablation,
 * App. A.6: per-token / per-channel symmetric quantization at more bits),
 * one code per byte:
 *   qmax = 2^(bits-1) - 1 (31 or 127), s = RN16(RN(RN(absmax * clip) / qmax)),
 *   q = clamp(rint_even(RN(y / s)), -qmax - 1, qmax) as int8.
 *   x fp16 [rows, n]; q int8 [rows, n]; scale fp16 [rows]; bits 6 or 8.
 * rotate != 0 needs n supported by quarot_hadamard_factor; rotate == 0 needs
 * n a positive multiple of 8.  Used offline for the weights as well.
 */
quarot_status quarot_quant_int8(const quarot_f16 *x, int8_t *q, quarot_f16 *scale, int64_t rows,
                                int64_t n, int rotate, float clip_ratio, int bits, void *stream);

/*
 * W8A8 GEMM with fused dequant (6- or 8-bit codes, one per byte):
 *   xq int8 [M, K], sx fp16 [M]; wq int8 [N, K], sw fp16 [N];
 *   y fp16 [M, N] = RN16(RN(RN(float(acc) * sx[m]) * sw[n])), acc exact int32;
 *   acc_out int32 [M, N] or NULL.
 * M, N >= 0; K a positive multiple of 64, at most 65536.
 */
quarot_status quarot_w8a8_gemm(const int8_t *xq, const quarot_f16 *sx, const int8_t *wq,
                               const quarot_f16 *sw, quarot_f16 *y, int32_t *acc_out,
                               int64_t M, int64_t N, int64_t K, void *stream);

/* Workspace of quarot_linear_w8a8: M*K code bytes and 2*M scale bytes, each
 * rounded up to 256 bytes (0 for invalid sizes).  Host-only. */
size_t quarot_linear_w8a8_workspace_size(int64_t M, int64_t K);

/*
 * The 6/8-bit linear layer: quarot_quant_int8(x, rotate, clip_ratio, bits)
 * into the workspace, then quarot_w8a8_gemm into y (two launches).  The
 * weights wq, sw come from quarot_quant_int8 of W [N, K] with the same
 * rotate and bits.  Size and alignment rules of both calls apply.
 */
quarot_status quarot_linear_w8a8(const quarot_f16 *x, const int8_t *wq, const quarot_f16 *sw,
                                 quarot_f16 *y, int64_t M, int64_t N, int64_t K, int rotate,
                                 float clip_ratio, int bits, void *workspace,
                                 size_t workspace_bytes, void *stream);

/*
 * Offline weight quantization with a per-row (per output channel) clip
 * search (§5 Setup: per-channel round-to-nearest weights whose clipping
 * ratio is picked by a linear search on the squared error; App. A.2).  For
 * each row y (w rotated like an activation row when rotate != 0) and each
 * candidate c_j = RN32((100 - j) / 100), j < n_candidates: the symmetric
 * quantizer of quarot_quant_int4 (bits = 4) or quarot_quant_int8 (6, 8)
 * with clip c_j, the terms e_i = RN64((y_i - q_i * s)^2) (the difference
 * exact in binary64), and E_j = their sum in this fixed binary64 order:
 * 256 interleaved partial sums P_t = e_t + e_{t+256} + ... (from +0, in
 * increasing i), then P_t += P_{t+h} for h = 128, 64, ..., 1; E_j = P_0.
 * The row keeps the first j with the smallest E_j; the codes and scale are
 * exactly those of the plain quantizer with clip c_best.
 *   w fp16 [rows, n]; q: uint8 [rows, n/2] (bits 4) or int8 [rows, n];
 *   scale fp16 [rows]; clip_out float32 [rows] (c_best);
 *   workspace: quarot_quant_search_workspace_size(rows, n, rotate) bytes
 *   (binary32 rotated rows; 0 without rotation), 16-byte aligned.
 * 1 <= n_candidates <= 100.
 */
size_t quarot_quant_search_workspace_size(int64_t rows, int64_t n, int rotate);
quarot_status quarot_quant_search(const quarot_f16 *w, void *q, quarot_f16 *scale,
                                  float *clip_out, int64_t rows, int64_t n, int rotate, int bits,
                                  int n_candidates, void *workspace, size_t workspace_bytes,
                                  void *stream);

/*
 * Group-wise quantization (§5.3, the group-size ablation of W4A4: a scale
 * per group of `group` consecutive input channels).  Each row (rotated by
 * H_n first when rotate != 0, kept in binary32) is cut into n / group
 * groups; each group is quantized exactly as quarot_quant_int4 quantizes a
 * whole row (its own absmax, s16 = RN16(absmax * clip_ratio / 7), codes
 * clamp(rint(y / s16), -8, 7)).
 *   x fp16 [rows, n]; q uint8 [rows, n/2] (packed as quarot_quant_int4);
 *   scale fp16 GROUP-MAJOR [n / group, rows]: scale[g * rows + r];
 *   workspace: quarot_quant_int4_grouped_workspace_size(rows, n, rotate)
 *   bytes (the binary32 rotated rows; 0 without rotation), 16-B aligned.
 * group: a power of two in [8, 512] dividing n.  Two launches with
 * rotation (rotate to binary32, then quantize), one without.
 */
size_t quarot_quant_int4_grouped_workspace_size(int64_t rows, int64_t n, int rotate);
quarot_status quarot_quant_int4_grouped(const quarot_f16 *x, uint8_t *q, quarot_f16 *scale,
                                        int64_t rows, int64_t n, int64_t group, int rotate,
                                        float clip_ratio, void *workspace,
                                        size_t workspace_bytes, void *stream);

/*
 * Group-wise W4A4 product (§5.3 group-size ablation; the per-token dequant
 * of §4 Stage 2b applied per group).  For each group g of `group` columns
 * of K: acc_g = exact int32 dot product of the codes,
 * t_g = RN(RN(f32(acc_g) * sx[g][m]) * sw[g][n]), and
 * y[m][n] = RN16(((+0 + t_0) + t_1) + ... ) in increasing g, in binary32.
 *   xq uint8 [M, K/2], wq uint8 [N, K/2] (packed int4 codes);
 *   sx fp16 [K/group, M], sw fp16 [K/group, N] (group-major, as written by
 *   quarot_quant_int4_grouped); y fp16 [M, N].
 * group: 64, 128 or 256; K a multiple of max(group, 128), K <= 65536.
 * One launch.
 */
quarot_status quarot_w4a4_gemm_grouped(const uint8_t *xq, const quarot_f16 *sx,
                                       const uint8_t *wq, const quarot_f16 *sw, quarot_f16 *y,
                                       int64_t M, int64_t N, int64_t K, int64_t group,
                                       void *stream);

/*
 * quarot_w4a4_gemm_grouped on operands in the tiled e3m2 layout of
 * quarot_pack_e3m2 (xq6 [K/128, M*96], wq6 [K/128, N*96]; the same int4
 * codes, each stored as the e3m2 number of its value): the same y, bit for
 * bit, from the fp6 matrix instruction (each group's sum of code products
 * is exact in binary32, so f32(acc_g) is that sum).
 * group: 128 or 256 (64 is QUAROT_ERR_UNSUPPORTED_SIZE: one instruction
 * spans 128 k); M and N multiples of 8; K a multiple of group,
 * K <= 65536.  One launch.
 */
quarot_status quarot_w4a4_gemm_grouped_e3m2(const uint8_t *xq6, const quarot_f16 *sx,
                                            const uint8_t *wq6, const quarot_f16 *sw,
                                            quarot_f16 *y, int64_t M, int64_t N, int64_t K,
                                            int64_t group, void *stream);

/*
 * The group-wise linear layer: quarot_quant_int4_grouped of x [M, K] into
 * the workspace, then quarot_w4a4_gemm_grouped.  wq, sw come from
 * quarot_quant_int4_grouped of W [N, K] with the same group and rotate.
 * workspace: quarot_linear_w4a4_grouped_workspace_size(M, K, group, rotate)
 * bytes, 256-B aligned (codes, then scales, then binary32 rotated rows).
 */
size_t quarot_linear_w4a4_grouped_workspace_size(int64_t M, int64_t K, int64_t group,
                                                 int rotate);
quarot_status quarot_linear_w4a4_grouped(const quarot_f16 *x, const uint8_t *wq,
                                         const quarot_f16 *sw, quarot_f16 *y, int64_t M,
                                         int64_t N, int64_t K, int64_t group, int rotate,
                                         float clip_ratio, void *workspace,
                                         size_t workspace_bytes, void *stream);

/*
 * The elementwise SwiGLU product alone: h = RN16(RN(silu(gate) * up)) with
 * the binary32 silu recipe of quarot_swiglu_quant_int4 below.
 * gate, up, h fp16 [count]; count a multiple of 8 (0 is a no-op).
 */
quarot_status quarot_swiglu(const quarot_f16 *gate, const quarot_f16 *up, quarot_f16 *h,
                            int64_t count, void *stream);

/*
 * The down-projection input of a SwiGLU FFN, rotated and quantized in one
 * launch (§4 Stage 1b: the online Hadamard sits between silu(gate) * up
 * and the 4-bit W_down):
 *   h = RN16(RN(silu(gate) * up)) elementwise, then exactly
 *   quarot_quant_int4(h, rotate = 1, clip_ratio), without storing h.
 * silu is binary32 by a fixed sequence of IEEE operations, so that its
 * result is reproducible (a Cody-Waite reduced exp, Taylor degree 7):
 *   x = clamp(-g, -88, 88), kf = rint_even(RN(x * RN32(1/ln 2))),
 *   r = fma(-kf, LN2_HI, x), r = fma(-kf, LN2_LO, r),
 *   p = 1 + r(1 + r(1/2! + r(1/3! + ... + r/7!))) by fma (RN32 coefficients),
 *   silu(g) = RN(g / RN(1 + ldexp(p, kf)))
 * with LN2_HI = 0x1.62e4p-1, LN2_LO = 0x1.7f7d1cp-20 (within 4 binary32
 * ulps of g/(1+exp(-g)) for every fp16 g).
 *   gate, up fp16 [rows, n]; q uint8 [rows, n/2]; scale fp16 [rows];
 *   n supported by quarot_hadamard_factor; clip_ratio in (0, 1].
 */
quarot_status quarot_swiglu_quant_int4(const quarot_f16 *gate, const quarot_f16 *up, uint8_t *q,
                                       quarot_f16 *scale, int64_t rows, int64_t n,
                                       float clip_ratio, void *stream);

/*
 * quarot_swiglu_quant_int4 with the codes in the tiled e3m2 layout (for
 * quarot_w4a4_gemm_e3m2); n as for quarot_quant_int4_e3m2 with rotation.
 */
quarot_status quarot_swiglu_quant_e3m2(const quarot_f16 *gate, const quarot_f16 *up, uint8_t *q6,
                                       quarot_f16 *scale, int64_t rows, int64_t n,
                                       float clip_ratio, void *stream);

/*
 * Hadamard transform across attention heads (§4 Stage 1c: with the
 * per-head factor I (x) H_dh fused into W_v and W_out offline, the online
 * part before out_proj is z <- z (H_nh (x) I_dh)).  Rows z [rows, n] with
 * n = n_heads * head_dim, head-major (element h * head_dim + d):
 *   y = RN16(z (H_nh (x) I_dh) / sqrt(n_heads)), the Walsh-Hadamard
 *   butterflies over the head index (bit 0 first) in binary32, one
 *   multiply by RN32(1/sqrt(n_heads)); a zero output is +0.
 * n_heads a power of two >= 2, head_dim a power of two >= 8,
 * n <= 32768.  z == y (in place) is allowed.
 */
quarot_status quarot_hadamard_heads(const quarot_f16 *z, quarot_f16 *y, int64_t rows,
                                    int64_t n_heads, int64_t head_dim, void *stream);

/*
 * The out_proj input: the binary32 head-wise transform above quantized
 * per row (token) to symmetric int4 exactly as quarot_quant_int4 does
 * (scale from the row's absmax, codes by IEEE division by the stored fp16
 * scale).  q uint8 [rows, n/2], scale fp16 [rows]; sizes as above.
 */
quarot_status quarot_hadamard_heads_quant_int4(const quarot_f16 *z, uint8_t *q,
                                               quarot_f16 *scale, int64_t rows, int64_t n_heads,
                                               int64_t head_dim, float clip_ratio, void *stream);

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

/*
 * Append (App. A.10, decode step): quantize the new tokens' head vectors
 * exactly as quarot_kv_quant does and store them at token position pos of
 * caches laid out [rows, s_max, ...]:
 *   kv_new fp16 [rows, head_dim]        (rows = batch * kv heads)
 *   q_cache uint8 [rows, s_max, head_dim/2]
 *   scale_cache, zero_cache fp16 [rows, s_max, head_dim/group]
 * Only position pos of each row is written.  0 <= pos < s_max; other size
 * rules as quarot_kv_quant.
 */
quarot_status quarot_kv_append(const quarot_f16 *kv_new, uint8_t *q_cache,
                               quarot_f16 *scale_cache, quarot_f16 *zero_cache, int64_t rows,
                               int64_t s_max, int64_t pos, int64_t head_dim, int64_t group,
                               int rotate, float clip_ratio, void *stream);

/*
 * Bytes of device workspace quarot_kv_decode_attention needs for nq query
 * rows over seq_len tokens (0 when the sequence is not split).  Host-only.
 */
size_t quarot_kv_attention_workspace_size(int64_t nq, int64_t seq_len, int64_t head_dim);

/*
 * Decode attention over the 4-bit KV cache (§4 Stage 2c: fp16 queries,
 * the cache dequantized on the fly; App. A.10 "Decode").  The keys and
 * values are in the rotated basis and the queries are rotated alike (by
 * quarot_hadamard with n = head_dim), so q . khat is the attention score.
 *   q fp16 [nq, head_dim]; query row i reads cache row i / (nq / nkv)
 *   k_codes, v_codes uint8 [nkv, s_max, head_dim/2]
 *   k_scale, k_zero, v_scale, v_zero fp16 [nkv, s_max, head_dim/group]
 *   out fp16 [nq, head_dim]
 * With khat = code * scale + zero (per group) and tokens t < seq_len:
 *   out = RN16(softmax_t(sm_scale * q . khat_t) . vhat), computed with
 *   binary32 accumulation and a running-max softmax (a floating-point
 *   result: it agrees with the exact value to a stated tolerance, not bit
 *   for bit).
 * head_dim 64, 128 or 256; group a power of two with 32 <= group <=
 * head_dim; nq a multiple of nkv; 1 <= seq_len <= s_max; workspace of at
 * least quarot_kv_attention_workspace_size bytes (may be NULL when that
 * is 0), 16-byte aligned.
 */
quarot_status quarot_kv_decode_attention(const quarot_f16 *q, const uint8_t *k_codes,
                                         const quarot_f16 *k_scale, const quarot_f16 *k_zero,
                                         const uint8_t *v_codes, const quarot_f16 *v_scale,
                                         const quarot_f16 *v_zero, quarot_f16 *out, int64_t nq,
                                         int64_t nkv, int64_t s_max, int64_t seq_len,
                                         int64_t head_dim, int64_t group, float sm_scale,
                                         void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QUAROT_H */
