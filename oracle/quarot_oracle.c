/*
 * QuaRot W4A4 linear-layer hot path: plain, slow CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference that the GPU library
 * is checked against.  Only the test suite, the smoke check and the bench's
 * CPU-baseline leg may load it.  It shares no code, header, table or constant
 * generator with the HIP library: both sides build the Hadamard factors from
 * the same published constructions, independently.
 *
 * Paper: "QuaRot: Outlier-Free 4-Bit Inference in Rotated LLMs"
 * (Ashkboos et al., arXiv 2404.00456).
 *
 * Arithmetic is IEEE binary32 with round-to-nearest-even, because the paper
 * fixes the online Hadamard transform to FP32 (App. A.7) and its scales and
 * outputs to FP16 (§4 Stage 2b).  Build with -O2 -ffp-contract=off and no
 * fast-math, so that every written operation is one correctly rounded op.
 *
 * Conventions (readings of the paper where it is silent or ambiguous):
 *  - Row vectors: a token row x of width n is rotated as y = x . H_n / sqrt(n),
 *    matching the right-multiplications X <- XQ and Z <- Z(H (x) I) of §4.
 *  - H_n = H_{2^k} (x) H_m (§3.1), element index i = a*m + b with a in
 *    [0, 2^k) and b in [0, m): m is the fast index.
 *  - Evaluation order of the rotation (the paper is silent; fp32 addition is
 *    not associative, so the order is part of the definition):
 *      1. t_i = f32(x_i)
 *      2. m-factor: for each a and output column b',
 *         u[a*m+b'] = RN32( sum_b Hm[b][b'] * t[a*m+b] ), the sum taken
 *         exactly and rounded once.  For fp16 inputs every partial sum is a
 *         multiple of 2^-24 below 172 * 65504 < 2^24 in magnitude, so an
 *         fp64 accumulation (any order) is exact; it is done here left to
 *         right in fp64.
 *      3. FWHT over a, butterfly bit j = 0, 1, ..., k-1 in increasing order;
 *         for p with bit j clear and q = p + 2^j:
 *         (u_p, u_q) <- (RN(u_p + u_q), RN(u_p - u_q)).
 *      4. y = RN(u * c) with c = RN32(1/sqrt(n)); a zero y is +0 (the sign
 *         of a zero is not part of the result: y = RN(RN(u * c) + 0)).
 *  - Symmetric int4 (§4 Stage 2b, scale = absmax / 7):
 *      s32 = RN(RN(absmax * clip) / 7), s16 = RN16(s32), and the codes use
 *      the stored s16: q = clamp(rint_even(RN(y / f32(s16))), -8, 7);
 *      s16 == 0 gives all-zero codes.
 *  - Packing: byte j of a row holds element 2j in the low nibble and 2j+1 in
 *    the high nibble, two's complement.
 *  - Dequant: Y = RN16(RN(RN(f32(acc) * f32(sx)) * f32(sw))).
 *  - KV cache (§5 Setup: asymmetric, groups of 128, clip 0.95): per group
 *      mx' = RN(max*clip), mn' = RN(min*clip),
 *      s16 = RN16(RN(RN(mx' - mn') / 15)), z16 = RN16(mn'),
 *      q = clamp(rint_even(RN(RN(y - f32(z16)) / f32(s16))), 0, 15),
 *      dequant yhat = RN(RN(f32(q) * f32(s16)) + f32(z16)), optionally
 *      rotated back (H/sqrt(n) is an involution for symmetric Sylvester H),
 *      then RN16.
 *  - 6/8-bit variants (§5.3 RTN rows, App. A.6): the symmetric quantizer with
 *    qmax = 2^(bits-1) - 1 in place of 7, codes clamped to [-qmax-1, qmax],
 *    one signed byte each; int8 x int8 -> int32, dequant as above.
 *  - Weight clip search (§5 Setup, App. A.2): candidates
 *    c_j = RN32((100 - j) / 100), the error sum_i RN64((y_i - q_i s16)^2)
 *    with each difference exact, summed in a fixed order (256 interleaved
 *    partial sums, then a halving tree), the first j of least error.
 *  - Group-wise (§5.3 group-size ablation): each group of G channels of a
 *    (rotated) row quantized like a whole row, scales group-major [n/G, rows];
 *    the product sums t_g = RN(RN(f32(acc_g) sx_g) sw_g) over g in increasing
 *    order from +0 in binary32.
 *  - SwiGLU input (§4 Stage 1b): h = RN16(RN(silu(g) u)) with a fixed binary32
 *    silu (Cody-Waite reduction, degree-7 Taylor exp; see orc_silu_f32).
 *  - Decode attention (§4 Stage 2c): fp64 scores and softmax over the exactly
 *    dequantized cache, the output rounded once to fp16.
 *
 * Pins: every function here is checked by tests/test_oracle_*.py against
 * something other than itself (paper values, closed forms, brute force,
 * numpy/scipy/torch references, exact-rational searches).  Parity unpinned
 * (conventions with no external definition, fixed here and shared by the
 * GPU side): the binary32 order of the butterfly stages (checked exactly only
 * where no rounding occurs), which Hadamard matrix of each order m is used,
 * the silu recipe's exp (pinned to 4 ulps of the true exp), and the order of
 * the group-wise sum (pinned within its rounding bound).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_OK = 0, ORC_ERR_ARG = 1, ORC_ERR_SIZE = 2, ORC_ERR_NOMEM = 3 };

/* ------------------------------------------------------------------------ */
/* IEEE binary16 <-> binary32, written out from the format definitions.     */
/* ------------------------------------------------------------------------ */

float orc_f16_to_f32(uint16_t h)
{
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    uint32_t e = (h >> 10) & 0x1Fu;
    uint32_t man = h & 0x3FFu;
    uint32_t bits;
    float f;
    if (e == 0) {
        /* zero or subnormal: value = man * 2^-24, exact in binary32 */
        f = (float)man * 5.9604644775390625e-8f;
        return sign ? -f : f;
    }
    if (e == 31)
        bits = sign | 0x7F800000u | (man << 13);
    else
        bits = sign | ((e - 15u + 127u) << 23) | (man << 13);
    memcpy(&f, &bits, 4);
    return f;
}

uint16_t orc_f32_to_f16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    uint32_t sign = (u >> 16) & 0x8000u;
    uint32_t exp8 = (u >> 23) & 0xFFu;
    uint32_t man = u & 0x7FFFFFu;
    if (exp8 == 0xFF) /* inf or nan */
        return (uint16_t)(sign | 0x7C00u | (man ? (0x200u | (man >> 13)) : 0u));
    int e = (int)exp8 - 127 + 15; /* binary16 biased exponent */
    if (e >= 31)
        return (uint16_t)(sign | 0x7C00u);
    if (e <= 0) {
        /* result is subnormal or zero: m16 = round(mant * 2^(e-14)) */
        if (e < -10)
            return (uint16_t)sign;
        uint32_t mant = man | 0x800000u;
        int shift = 14 - e; /* 14 .. 24 */
        uint32_t m16 = mant >> shift;
        uint32_t rem = mant & ((1u << shift) - 1u);
        uint32_t half = 1u << (shift - 1);
        if (rem > half || (rem == half && (m16 & 1u)))
            m16++;
        return (uint16_t)(sign | m16);
    }
    uint32_t r = ((uint32_t)e << 10) | (man >> 13);
    uint32_t rem = man & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (r & 1u)))
        r++; /* a carry may reach the exponent, up to 0x7C00 = inf */
    return (uint16_t)(sign | r);
}

/* binary64 -> binary16, round to nearest even, straight from the binary64
 * encoding (one rounding; going through binary32 first could round twice). */
uint16_t orc_f64_to_f16(double d)
{
    uint64_t u;
    memcpy(&u, &d, 8);
    uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
    int exp11 = (int)((u >> 52) & 0x7FFu);
    uint64_t man = u & 0xFFFFFFFFFFFFFull;
    if (exp11 == 0x7FF) /* inf or nan */
        return (uint16_t)(sign | 0x7C00u | (man ? 0x200u : 0u));
    int e = exp11 - 1023 + 15; /* binary16 biased exponent */
    if (e >= 31)
        return (uint16_t)(sign | 0x7C00u);
    /* significand with the implicit bit: 53 bits (binary64 subnormals are
     * far below the binary16 range and go to zero with the e < -10 rule) */
    uint64_t mant = man | (exp11 ? (1ull << 52) : 0ull);
    int shift; /* bits dropped to reach the binary16 significand */
    uint32_t base;
    if (e <= 0) {
        if (e < -10)
            return sign;
        shift = 42 + (1 - e); /* subnormal: units of 2^-24 */
        base = 0;
    } else {
        shift = 42;
        base = (uint32_t)e << 10;
        mant &= (1ull << 52) - 1ull; /* the exponent field carries the implicit bit */
    }
    uint64_t kept = mant >> shift;
    uint64_t rem = mant & ((1ull << shift) - 1ull);
    uint64_t half = 1ull << (shift - 1);
    uint32_t r = base + (uint32_t)kept;
    if (rem > half || (rem == half && (r & 1u)))
        r++; /* a carry may reach the exponent, up to 0x7C00 = inf */
    return (uint16_t)(sign | r);
}

void orc_f64_to_f16_array(const double *d, uint16_t *h, int64_t n)
{
    for (int64_t i = 0; i < n; i++)
        h[i] = orc_f64_to_f16(d[i]);
}

void orc_f16_to_f32_array(const uint16_t *h, float *f, int64_t n)
{
    for (int64_t i = 0; i < n; i++)
        f[i] = orc_f16_to_f32(h[i]);
}

void orc_f32_to_f16_array(const float *f, uint16_t *h, int64_t n)
{
    for (int64_t i = 0; i < n; i++)
        h[i] = orc_f32_to_f16(f[i]);
}

/* ------------------------------------------------------------------------ */
/* Hadamard matrices (§3.1).                                                */
/* ------------------------------------------------------------------------ */

/* Sylvester: H_{2^k}[i][j] = (-1)^popcount(i & j), eq. (1) without the
 * 1/sqrt(2) per level (applied once, as c = 1/sqrt(n), at the end). */
int orc_sylvester_entry(int64_t i, int64_t j)
{
    return (__builtin_popcountll((unsigned long long)(i & j)) & 1) ? -1 : 1;
}

/* Legendre symbol of a modulo an odd prime p: 0, +1 or -1. */
static int legendre(int64_t a, int64_t p)
{
    a %= p;
    if (a < 0)
        a += p;
    if (a == 0)
        return 0;
    int64_t r = 1, b = a, e = (p - 1) / 2;
    while (e) {
        if (e & 1)
            r = r * b % p;
        b = b * b % p;
        e >>= 1;
    }
    return r == 1 ? 1 : -1;
}

/* Paley's first construction for a prime q = 3 mod 4: with the skew
 * Jacobsthal matrix Q[i][j] = chi(j - i) (chi the Legendre symbol),
 * S = [[0, 1^T], [-1, Q]] and H = I + S has order q + 1.
 * Used for m = 12 (q = 11), 20 (q = 19) and 108 (q = 107). */
static void paley1(int q, int8_t *H)
{
    const int n = q + 1;
    for (int r = 0; r < n; r++)
        for (int s = 0; s < n; s++) {
            int v;
            if (r == 0 && s == 0)
                v = 0;
            else if (r == 0)
                v = 1;
            else if (s == 0)
                v = -1;
            else
                v = legendre((s - 1) - (r - 1), q);
            H[r * n + s] = (int8_t)(v + (r == s ? 1 : 0));
        }
}

/* H_28 by Paley's second construction with q = 13 (q = 1 mod 4):
 * C = [[0, 1^T], [1, Q]] with the Jacobsthal matrix Q[i][j] = chi(j - i),
 * H = C (x) [[1, 1], [1, -1]] + I (x) [[1, -1], [-1, -1]]. */
static void paley2_28(int8_t *H)
{
    const int q = 13, n = 2 * (q + 1);
    for (int r = 0; r < q + 1; r++)
        for (int s = 0; s < q + 1; s++) {
            int c;
            if (r == 0 && s == 0)
                c = 0;
            else if (r == 0 || s == 0)
                c = 1;
            else
                c = legendre((s - 1) - (r - 1), q);
            for (int u = 0; u < 2; u++)
                for (int v = 0; v < 2; v++) {
                    int kron = c * ((u == 1 && v == 1) ? -1 : 1);
                    int diag = 0;
                    if (r == s)
                        diag = (u == 0 && v == 0) ? 1 : -1;
                    H[(2 * r + u) * n + (2 * s + v)] = (int8_t)(kron + diag);
                }
        }
}

/* H_172 by the Goethals-Seidel array over four circulants of order 43.
 * Each circulant's first row x is +-1 with x[0] given, and for j > 0
 * x[j] = -1 exactly when j lies in a chosen union of cyclotomic classes of
 * order 6 of Z_43, C_c = { 3^(6t + c) mod 43 }, 3 being a primitive root.
 *   A: x[0] = -1, classes {0, 1}
 *   B: x[0] = +1, classes {0, 1, 3}
 *   C: same as B
 *   D: x[0] = +1, classes {0, 2, 3}
 * Their periodic autocorrelations sum to zero off the origin, so with
 * circulant X[i][j] = x[(j - i) mod 43] and back-identity R,
 *   [ A    BR   CR   DR  ]
 *   [ -BR  A    D'R  -C'R]
 *   [ -CR  -D'R A    B'R ]
 *   [ -DR  C'R  -B'R A   ]
 * is Hadamard of order 172 (the check H H^T = 172 I is in the tests). */
static void gs_172(int8_t *H)
{
    const int p = 43, n = 172;
    int cls[43];
    cls[0] = -1;
    int v = 1;
    for (int t = 0; t < p - 1; t++) {
        cls[v] = t % 6;
        v = v * 3 % p;
    }
    const int first[4] = {-1, 1, 1, 1};
    const int member[4][6] = {
        {1, 1, 0, 0, 0, 0}, {1, 1, 0, 1, 0, 0}, {1, 1, 0, 1, 0, 0}, {1, 0, 1, 1, 0, 0}};
    int seq[4][43];
    for (int s = 0; s < 4; s++) {
        seq[s][0] = first[s];
        for (int j = 1; j < p; j++)
            seq[s][j] = member[s][cls[j]] ? -1 : 1;
    }
    /* block (I, J): which sequence, transposed?, times R?, sign */
    const int bseq[4][4] = {{0, 1, 2, 3}, {1, 0, 3, 2}, {2, 3, 0, 1}, {3, 2, 1, 0}};
    const int btr[4][4] = {{0, 0, 0, 0}, {0, 0, 1, 1}, {0, 1, 0, 1}, {0, 1, 1, 0}};
    const int bsign[4][4] = {{1, 1, 1, 1}, {-1, 1, 1, -1}, {-1, -1, 1, 1}, {-1, 1, -1, 1}};
    for (int I = 0; I < 4; I++)
        for (int J = 0; J < 4; J++) {
            const int *x = seq[bseq[I][J]];
            for (int i = 0; i < p; i++)
                for (int j = 0; j < p; j++) {
                    int e;
                    if (I == J) {
                        e = x[((j - i) % p + p) % p]; /* plain circulant A */
                    } else {
                        /* (X R)[i][j] = X[i][p-1-j]; (X^T R)[i][j] = X[p-1-j][i] */
                        int jj = p - 1 - j;
                        e = btr[I][J] ? x[((i - jj) % p + p) % p] : x[((jj - i) % p + p) % p];
                    }
                    H[(I * p + i) * n + (J * p + j)] = (int8_t)(bsign[I][J] * e);
                }
        }
}

/* Writes the m x m +-1 factor used for n = 2^k * m.  Returns ORC_OK, or
 * ORC_ERR_SIZE for an order without a compiled construction. */
int orc_hm_table(int m, int8_t *out)
{
    if (m == 1) {
        out[0] = 1;
        return ORC_OK;
    }
    if (m == 12 || m == 20 || m == 108) {
        paley1(m - 1, out);
        return ORC_OK;
    }
    if (m == 28) {
        paley2_28(out);
        return ORC_OK;
    }
    if (m == 172) {
        gs_172(out);
        return ORC_OK;
    }
    return ORC_ERR_SIZE;
}

/* n = 2^k * m with m in {1, 12, 20, 28, 108, 172}; the odd part of n picks m. */
int orc_hadamard_factor(int64_t n, int *log2_pow2, int *m_out)
{
    if (n <= 0)
        return ORC_ERR_ARG;
    static const int ms[6] = {1, 12, 20, 28, 108, 172};
    for (int t = 0; t < 6; t++) {
        int64_t m = ms[t];
        if (n % m)
            continue;
        int64_t p = n / m;
        if (p & (p - 1))
            continue;
        int k = 0;
        while ((1LL << k) < p)
            k++;
        *log2_pow2 = k;
        *m_out = (int)m;
        return ORC_OK;
    }
    return ORC_ERR_SIZE;
}

float orc_rotation_scale(int64_t n)
{
    return (float)(1.0 / sqrt((double)n));
}

/* ------------------------------------------------------------------------ */
/* Rotation (§3.1 Kronecker construction; §4 Stage 1b online Hadamard).     */
/* ------------------------------------------------------------------------ */

/* One row, fp32 in, fp32 out, canonical order (see header).  u is n floats
 * of scratch. */
static void rotate_row(const float *t, float *y, float *u, int64_t n, int k, int m,
                       const int8_t *Hm, float c)
{
    int64_t A = n / m;
    /* step 2: m-factor, u[a*m + b'] = RN32(sum_b Hm[b][b'] t[a*m + b]),
     * summed in fp64 (exact for fp16-valued t) and rounded once */
    for (int64_t a = 0; a < A; a++) {
        const float *ta = t + a * m;
        for (int bp = 0; bp < m; bp++) {
            double acc = 0.0;
            for (int b = 0; b < m; b++)
                acc = Hm[b * m + bp] > 0 ? acc + (double)ta[b] : acc - (double)ta[b];
            u[a * m + bp] = (float)acc;
        }
    }
    /* step 3: FWHT over a, bits low to high */
    for (int j = 0; j < k; j++) {
        int64_t h = 1LL << j;
        for (int64_t p = 0; p < A; p++) {
            if (p & h)
                continue;
            int64_t q = p + h;
            for (int b = 0; b < m; b++) {
                float up = u[p * m + b], uq = u[q * m + b];
                u[p * m + b] = up + uq;
                u[q * m + b] = up - uq;
            }
        }
    }
    /* step 4: one scale multiply; adding +0 turns a -0 into +0 and leaves
     * every other value as it is */
    for (int64_t i = 0; i < n; i++)
        y[i] = u[i] * c + 0.0f;
}

struct rot_plan {
    int k, m;
    float c;
    int8_t *Hm;
};

static int plan_init(struct rot_plan *pl, int64_t n)
{
    if (orc_hadamard_factor(n, &pl->k, &pl->m) != ORC_OK)
        return ORC_ERR_SIZE;
    pl->c = orc_rotation_scale(n);
    pl->Hm = (int8_t *)malloc((size_t)pl->m * pl->m);
    if (!pl->Hm)
        return ORC_ERR_NOMEM;
    orc_hm_table(pl->m, pl->Hm);
    return ORC_OK;
}

/* y[rows, n] (fp32) = rotation of t[rows, n] (fp32). */
int orc_rotate_f32(const float *t, float *y, int64_t rows, int64_t n)
{
    struct rot_plan pl;
    int st = plan_init(&pl, n);
    if (st)
        return st;
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *u = (float *)malloc((size_t)n * sizeof(float));
        if (!u) {
            err |= 1;
            continue;
        }
        rotate_row(t + r * n, y + r * n, u, n, pl.k, pl.m, pl.Hm, pl.c);
        free(u);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* fp16 in, fp32 rotated rows out. */
int orc_rotate_f16(const uint16_t *x, float *y, int64_t rows, int64_t n)
{
    struct rot_plan pl;
    int st = plan_init(&pl, n);
    if (st)
        return st;
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * 2 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(x[r * n + i]);
        rotate_row(t, y + r * n, t + n, n, pl.k, pl.m, pl.Hm, pl.c);
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* Standalone online Hadamard: y = RN16(rotation of x). */
int orc_hadamard_f16(const uint16_t *x, uint16_t *y, int64_t rows, int64_t n)
{
    float *tmp = (float *)malloc((size_t)rows * n * sizeof(float));
    if (!tmp)
        return ORC_ERR_NOMEM;
    int st = orc_rotate_f16(x, tmp, rows, n);
    if (st == ORC_OK)
        orc_f32_to_f16_array(tmp, y, rows * n);
    free(tmp);
    return st;
}

/* ------------------------------------------------------------------------ */
/* Symmetric per-token int4 quantization (§4 Stage 2b).                     */
/* ------------------------------------------------------------------------ */

static void quant_sym_row(const float *y, int64_t n, float clip, uint8_t *q, uint16_t *s)
{
    float amax = 0.0f;
    for (int64_t i = 0; i < n; i++) {
        float a = fabsf(y[i]);
        if (a > amax)
            amax = a;
    }
    float s32 = (amax * clip) / 7.0f;
    uint16_t s16 = orc_f32_to_f16(s32);
    float sf = orc_f16_to_f32(s16);
    *s = s16;
    for (int64_t j = 0; j < n / 2; j++) {
        int code[2];
        for (int h = 0; h < 2; h++) {
            int v = 0;
            if (sf != 0.0f) {
                float r = rintf(y[2 * j + h] / sf);
                if (r < -8.0f)
                    r = -8.0f;
                if (r > 7.0f)
                    r = 7.0f;
                v = (int)r;
            }
            code[h] = v & 0xF;
        }
        q[j] = (uint8_t)(code[0] | (code[1] << 4));
    }
}

/* fp32 rows -> packed int4 codes [rows, n/2] + fp16 scales [rows]. */
int orc_quant_sym_f32(const float *y, uint8_t *q, uint16_t *s, int64_t rows, int64_t n,
                      float clip)
{
    if (n <= 0 || (n & 1) || rows < 0)
        return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        quant_sym_row(y + r * n, n, clip, q + r * (n / 2), s + r);
    return ORC_OK;
}

/* fp16 rows -> (optional rotation, kept in fp32) -> packed int4 + scales. */
int orc_quant_int4(const uint16_t *x, uint8_t *q, uint16_t *s, int64_t rows, int64_t n,
                   int rotate, float clip)
{
    if (n <= 0 || (n & 1) || rows < 0)
        return ORC_ERR_ARG;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (rotate) {
        int st = plan_init(&pl, n);
        if (st)
            return st;
    }
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * 3 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(x[r * n + i]);
        const float *y = t;
        if (rotate) {
            rotate_row(t, t + n, t + 2 * n, n, pl.k, pl.m, pl.Hm, pl.c);
            y = t + n;
        }
        quant_sym_row(y, n, clip, q + r * (n / 2), s + r);
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Prologues of the two online-Hadamard sites of a layer (§4 Stage 1b: the  */
/* input of the FFN down-projection, silu(gate) * up; §4 Stage 1c: the      */
/* attention output before out_proj, rotated across heads).                 */
/* ------------------------------------------------------------------------ */

/* SiLU in binary32 by a fixed sequence of IEEE operations (so that every
 * implementation that performs the same operations gets the same bits):
 *   x  = clamp(-g, -88, 88)
 *   kf = rint_even(RN(x * log2(e)))
 *   r  = fma(-kf, LN2_HI, x); r = fma(-kf, LN2_LO, r)   (Cody-Waite reduction)
 *   p  = 1 + r (1 + r (1/2 + r (1/6 + ... + r/5040)))   (Taylor, Horner in fma)
 *   E  = p * 2^kf                                      (ldexp)
 *   silu(g) = RN(g / RN(1 + E))
 * E approximates exp(-g) to a few binary32 ulps; |r| <= ln(2)/2, where the
 * degree-7 Taylor remainder is below 2^-27. */
static const float ORC_LOG2E = 0x1.715476p+0f;   /* RN32(1 / ln 2) */
static const float ORC_LN2_HI = 0x1.62e4p-1f;     /* ln 2 to 16 bits: kf * LN2_HI is exact */
static const float ORC_LN2_LO = 0x1.7f7d1cp-20f;  /* RN32(ln 2 - LN2_HI) */
/* RN32(1/k!) for k = 7 .. 2 */
static const float ORC_C7 = 0x1.a01a02p-13f, ORC_C6 = 0x1.6c16c2p-10f, ORC_C5 = 0x1.111112p-7f,
                   ORC_C4 = 0x1.555556p-5f, ORC_C3 = 0x1.555556p-3f;

float orc_silu_f32(float g)
{
    float x = -g;
    if (x > 88.0f)
        x = 88.0f;
    if (x < -88.0f)
        x = -88.0f;
    float kf = rintf(x * ORC_LOG2E);
    float r = fmaf(-kf, ORC_LN2_HI, x);
    r = fmaf(-kf, ORC_LN2_LO, r);
    float p = ORC_C7;
    p = fmaf(p, r, ORC_C6);
    p = fmaf(p, r, ORC_C5);
    p = fmaf(p, r, ORC_C4);
    p = fmaf(p, r, ORC_C3);
    p = fmaf(p, r, 0.5f);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    float e = ldexpf(p, (int)kf);
    float den = 1.0f + e;
    return g / den;
}

/* h = RN16(RN(silu(g) * u)): the fp16 input of the down-projection. */
static uint16_t swiglu_one(uint16_t g, uint16_t u)
{
    float sg = orc_silu_f32(orc_f16_to_f32(g));
    return orc_f32_to_f16(sg * orc_f16_to_f32(u));
}

int orc_swiglu_f16(const uint16_t *gate, const uint16_t *up, uint16_t *h, int64_t n)
{
    if (n < 0)
        return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++)
        h[i] = swiglu_one(gate[i], up[i]);
    return ORC_OK;
}

/* The down-projection input, rotated and quantized per token: exactly
 * orc_quant_int4 of orc_swiglu_f16(gate, up). */
int orc_swiglu_quant_int4(const uint16_t *gate, const uint16_t *up, uint8_t *q, uint16_t *s,
                          int64_t rows, int64_t n, int rotate, float clip)
{
    if (n <= 0 || (n & 1) || rows < 0)
        return ORC_ERR_ARG;
    uint16_t *h = (uint16_t *)malloc((size_t)(rows * n) * 2 + 2);
    if (!h)
        return ORC_ERR_NOMEM;
    int st = orc_swiglu_f16(gate, up, h, rows * n);
    if (st == ORC_OK)
        st = orc_quant_int4(h, q, s, rows, n, rotate, clip);
    free(h);
    return st;
}

/* Hadamard across heads (§4 Stage 1c, "Hadamard heads"): a row z of width
 * nh * dh (head-major: element h*dh + d) becomes y = z (H_nh (x) I_dh) /
 * sqrt(nh).  For each d the Walsh-Hadamard butterflies run over the head
 * index h, bit 0 first, in binary32; then one multiply by RN32(1/sqrt(nh));
 * a zero y is +0.  nh must be a power of two. */
static void heads_row(const float *t, float *y, int64_t nh, int64_t dh, float c)
{
    for (int64_t i = 0; i < nh * dh; i++)
        y[i] = t[i];
    for (int64_t h = 1; h < nh; h <<= 1)
        for (int64_t p = 0; p < nh; p++) {
            if (p & h)
                continue;
            for (int64_t d = 0; d < dh; d++) {
                float up = y[p * dh + d], uq = y[(p + h) * dh + d];
                y[p * dh + d] = up + uq;
                y[(p + h) * dh + d] = up - uq;
            }
        }
    for (int64_t i = 0; i < nh * dh; i++)
        y[i] = y[i] * c + 0.0f;
}

static int heads_args(int64_t rows, int64_t nh, int64_t dh)
{
    if (rows < 0 || nh < 2 || dh < 1 || (nh & (nh - 1)))
        return ORC_ERR_ARG;
    return ORC_OK;
}

/* fp16 rows -> binary32 rotated rows [rows, nh*dh]. */
int orc_heads_f16(const uint16_t *z, float *y, int64_t rows, int64_t nh, int64_t dh)
{
    int st = heads_args(rows, nh, dh);
    if (st)
        return st;
    const int64_t n = nh * dh;
    const float c = orc_rotation_scale(nh);
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(z[r * n + i]);
        heads_row(t, y + r * n, nh, dh, c);
        free(t);
    }
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* The out_proj input rotated across heads and quantized per token
 * (symmetric int4, as orc_quant_sym_f32). */
int orc_heads_quant_int4(const uint16_t *z, uint8_t *q, uint16_t *s, int64_t rows, int64_t nh,
                         int64_t dh, float clip)
{
    int st = heads_args(rows, nh, dh);
    if (st)
        return st;
    if ((nh * dh) & 1)
        return ORC_ERR_ARG;
    float *y = (float *)malloc((size_t)(rows * nh * dh) * sizeof(float) + 4);
    if (!y)
        return ORC_ERR_NOMEM;
    st = orc_heads_f16(z, y, rows, nh, dh);
    if (st == ORC_OK)
        st = orc_quant_sym_f32(y, q, s, rows, nh * dh, clip);
    free(y);
    return st;
}

/* ------------------------------------------------------------------------ */
/* 6- and 8-bit variants (§5.3 RTN ablation, App. A.6: the same per-token / */
/* per-channel symmetric scheme at more bits), one code per byte.           */
/* ------------------------------------------------------------------------ */

/* qmax = 2^(bits-1) - 1:  s16 = RN16(RN(RN(absmax * clip) / qmax)),
 * q = clamp(rint_even(RN(y / f32(s16))), -qmax - 1, qmax); s16 == 0 gives
 * codes 0. */
static void quant_sym8_row(const float *y, int64_t n, float clip, int qmax, int8_t *q,
                           uint16_t *s)
{
    float amax = 0.0f;
    for (int64_t i = 0; i < n; i++) {
        float a = fabsf(y[i]);
        if (a > amax)
            amax = a;
    }
    float s32 = (amax * clip) / (float)qmax;
    uint16_t s16 = orc_f32_to_f16(s32);
    float sf = orc_f16_to_f32(s16);
    *s = s16;
    for (int64_t i = 0; i < n; i++) {
        int v = 0;
        if (sf != 0.0f) {
            float r = rintf(y[i] / sf);
            if (r < (float)(-qmax - 1))
                r = (float)(-qmax - 1);
            if (r > (float)qmax)
                r = (float)qmax;
            v = (int)r;
        }
        q[i] = (int8_t)v;
    }
}

int orc_quant_sym8_f32(const float *y, int8_t *q, uint16_t *s, int64_t rows, int64_t n,
                       float clip, int bits)
{
    if (n <= 0 || rows < 0 || (bits != 6 && bits != 8))
        return ORC_ERR_ARG;
    const int qmax = (1 << (bits - 1)) - 1;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++)
        quant_sym8_row(y + r * n, n, clip, qmax, q + r * n, s + r);
    return ORC_OK;
}

/* fp16 rows -> (optional rotation, kept in fp32) -> int8 codes [rows, n]. */
int orc_quant_int8(const uint16_t *x, int8_t *q, uint16_t *s, int64_t rows, int64_t n,
                   int rotate, float clip, int bits)
{
    if (n <= 0 || rows < 0 || (bits != 6 && bits != 8))
        return ORC_ERR_ARG;
    const int qmax = (1 << (bits - 1)) - 1;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (rotate) {
        int st = plan_init(&pl, n);
        if (st)
            return st;
    }
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * 3 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(x[r * n + i]);
        const float *y = t;
        if (rotate) {
            rotate_row(t, t + n, t + 2 * n, n, pl.k, pl.m, pl.Hm, pl.c);
            y = t + n;
        }
        quant_sym8_row(y, n, clip, qmax, q + r * n, s + r);
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* Sum of e[0..n) in the fixed binary64 order that defines the clip
 * search's error (the paper gives no order, and binary64 addition is not
 * associative): 256 interleaved partial sums P_t = e_t + e_{t+256} + ...,
 * each from +0 in increasing index, then halved pairwise,
 * P_t <- P_t + P_{t+h} for h = 128, 64, ..., 1; the result is P_0. */
static double search_err_sum(const double *e, int64_t n)
{
    double P[256];
    for (int t = 0; t < 256; t++)
        P[t] = 0.0;
    for (int64_t i = 0; i < n; i++)
        P[i % 256] = P[i % 256] + e[i];
    for (int h = 128; h >= 1; h /= 2)
        for (int t = 0; t < h; t++)
            P[t] = P[t] + P[t + h];
    return P[0];
}

/* Weight quantization with a per-row clipping search (§5 Setup: per-channel
 * round-to-nearest weights whose clipping ratio is picked by a linear search
 * on the squared error; App. A.2).  For each row (output channel) y
 * (rotated if asked), candidates c_j = RN32((100 - j) / 100), j < ncand; for
 * each the scale and codes of the symmetric quantizer with that clip, the
 * terms e_i = RN64(d_i^2) with d_i = y_i - q_i s16 (exact in binary64), and
 * E_j = search_err_sum(e).  The row keeps the first j with the smallest E_j.
 * bits = 4 packs nibbles, 6 or 8 stores one code per byte.
 * clip_out[r] = c_best. */
int orc_quant_search(const uint16_t *x, void *q, uint16_t *s, float *clip_out, int64_t rows,
                     int64_t n, int rotate, int bits, int ncand)
{
    if (n <= 0 || (n & 1) || rows < 0 || ncand < 1 || ncand > 100 ||
        (bits != 4 && bits != 6 && bits != 8))
        return ORC_ERR_ARG;
    const int qmax = (1 << (bits - 1)) - 1;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (rotate) {
        int st = plan_init(&pl, n);
        if (st)
            return st;
    }
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * 3 * sizeof(float));
        double *et = (double *)malloc((size_t)n * sizeof(double));
        if (!t || !et) {
            free(t);
            free(et);
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(x[r * n + i]);
        const float *y = t;
        if (rotate) {
            rotate_row(t, t + n, t + 2 * n, n, pl.k, pl.m, pl.Hm, pl.c);
            y = t + n;
        }
        float amax = 0.0f;
        for (int64_t i = 0; i < n; i++)
            if (fabsf(y[i]) > amax)
                amax = fabsf(y[i]);
        double best_e = INFINITY;
        float best_c = 1.0f;
        for (int j = 0; j < ncand; j++) {
            const float c = (float)((double)(100 - j) / 100.0);
            const uint16_t s16 = orc_f32_to_f16((amax * c) / (float)qmax);
            const float sf = orc_f16_to_f32(s16);
            for (int64_t i = 0; i < n; i++) {
                int v = 0;
                if (sf != 0.0f) {
                    float rr = rintf(y[i] / sf);
                    if (rr < (float)(-qmax - 1))
                        rr = (float)(-qmax - 1);
                    if (rr > (float)qmax)
                        rr = (float)qmax;
                    v = (int)rr;
                }
                const double d = (double)y[i] - (double)v * (double)sf;
                et[i] = d * d;
            }
            const double e = search_err_sum(et, n);
            if (e < best_e) {
                best_e = e;
                best_c = c;
            }
        }
        clip_out[r] = best_c;
        if (bits == 4)
            quant_sym_row(y, n, best_c, (uint8_t *)q + r * (n / 2), s + r);
        else
            quant_sym8_row(y, n, best_c, qmax, (int8_t *)q + r * n, s + r);
        free(t);
        free(et);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* acc[M, N] = Xq[M, K] . Wq[N, K]^T over int8 codes, exact in int32
 * (|acc| <= 128^2 K). */
int orc_gemm_i8(const int8_t *xq, const int8_t *wq, int32_t *acc, int64_t M, int64_t N,
                int64_t K)
{
    if (K <= 0 || M < 0 || N < 0)
        return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; m++)
        for (int64_t n = 0; n < N; n++) {
            int32_t s = 0;
            for (int64_t k = 0; k < K; k++)
                s += (int32_t)xq[m * K + k] * (int32_t)wq[n * K + k];
            acc[m * N + n] = s;
        }
    return ORC_OK;
}

static int nibble(const uint8_t *row, int64_t k)
{
    int v = (row[k >> 1] >> ((k & 1) * 4)) & 0xF;
    return v >= 8 ? v - 16 : v;
}

/* ------------------------------------------------------------------------ */
/* Group-wise W4A4 (§5.3 group-wise ablation: a scale per group of G        */
/* consecutive input channels, for the activations and the weights).        */
/* ------------------------------------------------------------------------ */

/* Each (rotated) row in groups of G consecutive elements, each group
 * quantized exactly like a row of quant_sym_row (its own absmax and fp16
 * scale).  Codes [rows, n/2] as usual; scales group-major: s[g * rows + r]. */
int orc_quant_int4_grouped(const uint16_t *x, uint8_t *q, uint16_t *s, int64_t rows, int64_t n,
                           int64_t G, int rotate, float clip)
{
    if (n <= 0 || rows < 0 || G <= 0 || (G & 1) || n % G)
        return ORC_ERR_ARG;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (rotate) {
        int st = plan_init(&pl, n);
        if (st)
            return st;
    }
    const int64_t ng = n / G;
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)n * 3 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < n; i++)
            t[i] = orc_f16_to_f32(x[r * n + i]);
        const float *y = t;
        if (rotate) {
            rotate_row(t, t + n, t + 2 * n, n, pl.k, pl.m, pl.Hm, pl.c);
            y = t + n;
        }
        for (int64_t g = 0; g < ng; g++)
            quant_sym_row(y + g * G, G, clip, q + r * (n / 2) + g * (G / 2), s + g * rows + r);
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* The group-wise product: per group g of G columns of K, acc_g exact in
 * int32 and t_g = RN(RN(f32(acc_g) * sx[g][m]) * sw[g][n]) (the per-token
 * dequant of §4 Stage 2b, per group); Y = RN16 of the binary32 sum
 * ((+0 + t_0) + t_1) + ..., in increasing g.  sx [K/G, M], sw [K/G, N]. */
int orc_gemm_grouped(const uint8_t *xq, const uint16_t *sx, const uint8_t *wq, const uint16_t *sw,
                     uint16_t *y, int64_t M, int64_t N, int64_t K, int64_t G)
{
    if (K <= 0 || (K & 1) || M < 0 || N < 0 || G <= 0 || K % G)
        return ORC_ERR_ARG;
    const int64_t ng = K / G;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; m++) {
        const uint8_t *xr = xq + m * (K / 2);
        for (int64_t n = 0; n < N; n++) {
            const uint8_t *wr = wq + n * (K / 2);
            float sum = 0.0f;
            for (int64_t g = 0; g < ng; g++) {
                int32_t a = 0;
                for (int64_t k = g * G; k < (g + 1) * G; k++)
                    a += nibble(xr, k) * nibble(wr, k);
                float t = (float)a * orc_f16_to_f32(sx[g * M + m]);
                t = t * orc_f16_to_f32(sw[g * N + n]);
                sum = sum + t;
            }
            y[m * N + n] = orc_f32_to_f16(sum);
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Integer GEMM and dequantization (§4 Stage 2b, App. A.10).                */
/* ------------------------------------------------------------------------ */

/* acc[M, N] = Xq[M, K] . Wq[N, K]^T, exact in int32 (|acc| <= 64 K). */
int orc_gemm_i32(const uint8_t *xq, const uint8_t *wq, int32_t *acc, int64_t M, int64_t N,
                 int64_t K)
{
    if (K <= 0 || (K & 1) || M < 0 || N < 0)
        return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; m++) {
        const uint8_t *xr = xq + m * (K / 2);
        for (int64_t n = 0; n < N; n++) {
            const uint8_t *wr = wq + n * (K / 2);
            int32_t s = 0;
            for (int64_t k = 0; k < K; k++)
                s += nibble(xr, k) * nibble(wr, k);
            acc[m * N + n] = s;
        }
    }
    return ORC_OK;
}

/* Y[M, N] = RN16(RN(RN(f32(acc) * f32(sx[m])) * f32(sw[n]))). */
int orc_dequant(const int32_t *acc, const uint16_t *sx, const uint16_t *sw, uint16_t *y,
                int64_t M, int64_t N)
{
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; m++) {
        float a = orc_f16_to_f32(sx[m]);
        for (int64_t n = 0; n < N; n++) {
            float t = (float)acc[m * N + n] * a;
            y[m * N + n] = orc_f32_to_f16(t * orc_f16_to_f32(sw[n]));
        }
    }
    return ORC_OK;
}

/* The whole layer: quantize (optionally rotating) x, integer GEMM against
 * prepared weights, dequantize.  acc_out may be NULL. */
int orc_linear(const uint16_t *x, const uint8_t *wq, const uint16_t *sw, uint16_t *y,
               int32_t *acc_out, int64_t M, int64_t N, int64_t K, int rotate, float clip)
{
    uint8_t *xq = (uint8_t *)malloc((size_t)(M * K / 2) + 1);
    uint16_t *sx = (uint16_t *)malloc((size_t)M * 2 + 2);
    int32_t *acc = acc_out ? acc_out : (int32_t *)malloc((size_t)M * N * 4 + 4);
    int st = ORC_ERR_NOMEM;
    if (xq && sx && acc) {
        st = orc_quant_int4(x, xq, sx, M, K, rotate, clip);
        if (st == ORC_OK)
            st = orc_gemm_i32(xq, wq, acc, M, N, K);
        if (st == ORC_OK)
            st = orc_dequant(acc, sx, sw, y, M, N);
    }
    free(xq);
    free(sx);
    if (!acc_out)
        free(acc);
    return st;
}

/* ------------------------------------------------------------------------ */
/* 4-bit KV cache (§4 Stage 1d/2c, §5 Setup: asymmetric, group 128).        */
/* ------------------------------------------------------------------------ */

static void kv_quant_row(const float *y, int64_t D, int64_t G, float clip, uint8_t *q,
                         uint16_t *scale, uint16_t *zero)
{
    for (int64_t g = 0; g < D / G; g++) {
        const float *yg = y + g * G;
        float mx = yg[0], mn = yg[0];
        for (int64_t i = 1; i < G; i++) {
            if (yg[i] > mx)
                mx = yg[i];
            if (yg[i] < mn)
                mn = yg[i];
        }
        float mxc = mx * clip, mnc = mn * clip;
        float s32 = (mxc - mnc) / 15.0f;
        uint16_t s16 = orc_f32_to_f16(s32);
        uint16_t z16 = orc_f32_to_f16(mnc);
        float sf = orc_f16_to_f32(s16), zf = orc_f16_to_f32(z16);
        scale[g] = s16;
        zero[g] = z16;
        for (int64_t i = 0; i < G; i++) {
            int v = 0;
            if (sf != 0.0f) {
                float r = rintf((yg[i] - zf) / sf);
                if (r < 0.0f)
                    r = 0.0f;
                if (r > 15.0f)
                    r = 15.0f;
                v = (int)r;
            }
            int64_t e = g * G + i;
            if (e & 1)
                q[e >> 1] = (uint8_t)(q[e >> 1] | (v << 4));
            else
                q[e >> 1] = (uint8_t)v;
        }
    }
}

/* kv[rows, D] fp16 -> q[rows, D/2] (unsigned nibbles), scale/zero
 * [rows, D/G] fp16.  rotate applies H_D / sqrt(D) to each row first. */
int orc_kv_quant(const uint16_t *kv, uint8_t *q, uint16_t *scale, uint16_t *zero, int64_t rows,
                 int64_t D, int64_t G, int rotate, float clip)
{
    if (D <= 0 || (D & 1) || G <= 0 || (G & 1) || D % G || rows < 0)
        return ORC_ERR_ARG;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (rotate) {
        int st = plan_init(&pl, D);
        if (st)
            return st;
    }
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)D * 3 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < D; i++)
            t[i] = orc_f16_to_f32(kv[r * D + i]);
        const float *y = t;
        if (rotate) {
            rotate_row(t, t + D, t + 2 * D, D, pl.k, pl.m, pl.Hm, pl.c);
            y = t + D;
        }
        kv_quant_row(y, D, G, clip, q + r * (D / 2), scale + r * (D / G), zero + r * (D / G));
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* Inverse of the above up to quantization error: out[rows, D] fp16.
 * inverse_rotate applies H_D / sqrt(D) to the fp32 dequantized row before
 * the final RN16 (the Sylvester rotation is its own inverse). */
int orc_kv_dequant(const uint8_t *q, const uint16_t *scale, const uint16_t *zero, uint16_t *out,
                   int64_t rows, int64_t D, int64_t G, int inverse_rotate)
{
    if (D <= 0 || (D & 1) || G <= 0 || (G & 1) || D % G || rows < 0)
        return ORC_ERR_ARG;
    struct rot_plan pl = {0, 1, 1.0f, NULL};
    if (inverse_rotate) {
        int st = plan_init(&pl, D);
        if (st)
            return st;
        if (pl.m != 1) {
            free(pl.Hm);
            return ORC_ERR_SIZE;
        }
    }
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        float *t = (float *)malloc((size_t)D * 3 * sizeof(float));
        if (!t) {
            err |= 1;
            continue;
        }
        for (int64_t i = 0; i < D; i++) {
            int v = (q[r * (D / 2) + (i >> 1)] >> ((i & 1) * 4)) & 0xF;
            float sf = orc_f16_to_f32(scale[r * (D / G) + i / G]);
            float zf = orc_f16_to_f32(zero[r * (D / G) + i / G]);
            t[i] = (float)v * sf + zf;
        }
        const float *y = t;
        if (inverse_rotate) {
            rotate_row(t, t + D, t + 2 * D, D, pl.k, pl.m, pl.Hm, pl.c);
            y = t + D;
        }
        for (int64_t i = 0; i < D; i++)
            out[r * D + i] = orc_f32_to_f16(y[i]);
        free(t);
    }
    free(pl.Hm);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* Append (App. A.10, decode): quantize rows new tokens' head vectors and
 * store them at token position pos of a cache laid out [rows, s_max, ...]. */
int orc_kv_append(const uint16_t *kv, uint8_t *qc, uint16_t *sc, uint16_t *zc, int64_t rows,
                  int64_t s_max, int64_t pos, int64_t D, int64_t G, int rotate, float clip)
{
    if (rows < 0 || s_max <= 0 || pos < 0 || pos >= s_max)
        return ORC_ERR_ARG;
    uint8_t *q = (uint8_t *)malloc((size_t)(rows * D / 2) + 1);
    uint16_t *s = (uint16_t *)malloc((size_t)(rows * (D / G)) * 2 + 2);
    uint16_t *z = (uint16_t *)malloc((size_t)(rows * (D / G)) * 2 + 2);
    int st = ORC_ERR_NOMEM;
    if (q && s && z) {
        st = orc_kv_quant(kv, q, s, z, rows, D, G, rotate, clip);
        if (st == ORC_OK)
            for (int64_t r = 0; r < rows; r++) {
                memcpy(qc + (r * s_max + pos) * (D / 2), q + r * (D / 2), (size_t)(D / 2));
                memcpy(sc + (r * s_max + pos) * (D / G), s + r * (D / G), (size_t)(D / G) * 2);
                memcpy(zc + (r * s_max + pos) * (D / G), z + r * (D / G), (size_t)(D / G) * 2);
            }
    }
    free(q);
    free(s);
    free(z);
    return st;
}

/* Decode attention over the 4-bit cache (§4 Stage 2c, App. A.10): for query
 * row i (its cache row is i / (nq / nkv)), with the dequantized cache
 * khat[t][d] = code * scale + zero of the group of d (the rotated basis; the
 * queries are rotated alike, so q . khat is the attention score):
 *   score_t = sm_scale * sum_d q[d] khat[t][d],   t < seq_len
 *   p = softmax(score),  out[d] = RN16(sum_t p_t vhat[t][d]).
 * Everything is evaluated in fp64 (exact dequantization, plain softmax with
 * the maximum subtracted). */
int orc_kv_attention(const uint16_t *q, const uint8_t *kc, const uint16_t *ks,
                     const uint16_t *kz, const uint8_t *vc, const uint16_t *vs,
                     const uint16_t *vz, uint16_t *out, int64_t nq, int64_t nkv, int64_t s_max,
                     int64_t seq_len, int64_t D, int64_t G, float sm_scale)
{
    if (nq < 0 || nkv <= 0 || (nq % nkv) || s_max <= 0 || seq_len <= 0 || seq_len > s_max ||
        D <= 0 || (D & 1) || G <= 0 || D % G)
        return ORC_ERR_ARG;
    const int64_t rep = nq / nkv, ng = D / G;
    int err = 0;
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t i = 0; i < nq; i++) {
        const int64_t kv = i / rep;
        double *sc = (double *)malloc((size_t)seq_len * sizeof(double));
        double *o = (double *)malloc((size_t)D * sizeof(double));
        if (!sc || !o) {
            free(sc);
            free(o);
            err |= 1;
            continue;
        }
        double mx = -INFINITY;
        for (int64_t t = 0; t < seq_len; t++) {
            const int64_t row = kv * s_max + t;
            double acc = 0.0;
            for (int64_t d = 0; d < D; d++) {
                int c = (kc[row * (D / 2) + d / 2] >> ((d & 1) * 4)) & 0xF;
                double kh = (double)c * orc_f16_to_f32(ks[row * ng + d / G]) +
                            orc_f16_to_f32(kz[row * ng + d / G]);
                acc += (double)orc_f16_to_f32(q[i * D + d]) * kh;
            }
            sc[t] = acc * (double)sm_scale;
            if (sc[t] > mx)
                mx = sc[t];
        }
        double l = 0.0;
        for (int64_t t = 0; t < seq_len; t++) {
            sc[t] = exp(sc[t] - mx);
            l += sc[t];
        }
        for (int64_t d = 0; d < D; d++)
            o[d] = 0.0;
        for (int64_t t = 0; t < seq_len; t++) {
            const int64_t row = kv * s_max + t;
            const double p = sc[t] / l;
            for (int64_t d = 0; d < D; d++) {
                int c = (vc[row * (D / 2) + d / 2] >> ((d & 1) * 4)) & 0xF;
                double vh = (double)c * orc_f16_to_f32(vs[row * ng + d / G]) +
                            orc_f16_to_f32(vz[row * ng + d / G]);
                o[d] += p * vh;
            }
        }
        for (int64_t d = 0; d < D; d++)
            out[i * D + d] = orc_f64_to_f16(o[d]);
        free(sc);
        free(o);
    }
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Threads (for timing the oracle as a CPU baseline).                       */
/* ------------------------------------------------------------------------ */

void orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
