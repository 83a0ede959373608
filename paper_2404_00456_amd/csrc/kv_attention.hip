// Decode attention over the 4-bit KV cache (§4 Stage 2c: queries stay fp16,
// the cache is dequantized on the fly; App. A.10 "Decode"), for gfx950.
//
// For query row i (cache row i / rep) and tokens t < seq_len:
//   khat[t][d] = code * scale + zero of the group of d (rotated basis),
//   score_t = sm_scale * q . khat_t,  out = softmax(score) . vhat  (fp16).
// The dot products use the group constants once per token:
//   q . khat_t = scale_t * sum_d q[d] code[d] + zero_t * sum_d q[d]
//   sum_t p_t vhat[t][d] = sum_t (p_t scale_t) code[t][d] + sum_t p_t zero_t
// with binary32 accumulation and an online (running-max) softmax.
//
// Layout: a wave reads 16 bytes of codes per lane, 32 head-dim elements of
// one token: D/32 lanes per token, 64 / (D/32) tokens per load.  Each lane
// keeps the query slice and the output accumulators of its 32 elements.
// A block (4 waves) covers one query row and one chunk of the sequence;
// with several chunks the partial (max, sum, o) go to a workspace and a
// second kernel combines them.  Groups must be at least 32 wide, so that a
// lane's 32 elements share one scale and zero.  Head_dim 128 with one group
// per row takes the matrix-core kernel further below instead.
#include <algorithm>

#include "common.hpp"

namespace quarot {
namespace {

constexpr int ATT_WAVES = 4;
constexpr int ATT_U = 2;  // loads per lane per iteration

template <int J>
__device__ __forceinline__ float lane_sum(float v)
{
    if constexpr (J <= 3)
        return v + lane_xor_dpp<J>(v);
    else {
        const float2 p = lane_pair_swap<J>(v);
        return p.x + p.y;
    }
}

// byte i of w as float (v_cvt_f32_ubyte*)
template <int I>
__device__ __forceinline__ float ubyte(uint32_t w)
{
    return (float)((w >> (8 * I)) & 0xFFu);
}

// The low and high nibbles of each byte of w, as bytes.  The values pass
// through an empty asm: knowing the masks, the compiler would otherwise
// split each into four byte extractions (v_bfe / v_and) before converting,
// instead of one v_cvt_f32_ubyte0..3 per byte.
__device__ __forceinline__ void nibble_bytes(uint32_t w, uint32_t &lo, uint32_t &hi)
{
    lo = w & 0x0F0F0F0Fu;
    hi = (w >> 4) & 0x0F0F0F0Fu;
    __asm__("" : "+v"(lo), "+v"(hi));
}

// sum over e of x[e] * code_e for the 32 codes of one 16-byte slice
// (element 2j in the low nibble of byte j)
__device__ __forceinline__ float dot_codes(const uint4 &c, const float *x)
{
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t lo, hi;
        nibble_bytes(w[i], lo, hi);
        acc = __builtin_fmaf(x[8 * i + 0], ubyte<0>(lo), acc);
        acc = __builtin_fmaf(x[8 * i + 1], ubyte<0>(hi), acc);
        acc = __builtin_fmaf(x[8 * i + 2], ubyte<1>(lo), acc);
        acc = __builtin_fmaf(x[8 * i + 3], ubyte<1>(hi), acc);
        acc = __builtin_fmaf(x[8 * i + 4], ubyte<2>(lo), acc);
        acc = __builtin_fmaf(x[8 * i + 5], ubyte<2>(hi), acc);
        acc = __builtin_fmaf(x[8 * i + 6], ubyte<3>(lo), acc);
        acc = __builtin_fmaf(x[8 * i + 7], ubyte<3>(hi), acc);
    }
    return acc;
}

// o[e] += w * code_e
__device__ __forceinline__ void axpy_codes(const uint4 &c, float w, float *o)
{
    const uint32_t v[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t lo, hi;
        nibble_bytes(v[i], lo, hi);
        o[8 * i + 0] = __builtin_fmaf(w, ubyte<0>(lo), o[8 * i + 0]);
        o[8 * i + 1] = __builtin_fmaf(w, ubyte<0>(hi), o[8 * i + 1]);
        o[8 * i + 2] = __builtin_fmaf(w, ubyte<1>(lo), o[8 * i + 2]);
        o[8 * i + 3] = __builtin_fmaf(w, ubyte<1>(hi), o[8 * i + 3]);
        o[8 * i + 4] = __builtin_fmaf(w, ubyte<2>(lo), o[8 * i + 4]);
        o[8 * i + 5] = __builtin_fmaf(w, ubyte<2>(hi), o[8 * i + 5]);
        o[8 * i + 6] = __builtin_fmaf(w, ubyte<3>(lo), o[8 * i + 6]);
        o[8 * i + 7] = __builtin_fmaf(w, ubyte<3>(hi), o[8 * i + 7]);
    }
}

// The block's waves combined (thread d < D owns output element d): each
// wave left its running maximum, its sum of weights and its unnormalized
// output (zero-point term included) in red[w].  The result is the output
// row, or the split's partial (max, sum, o).
template <int D>
__device__ __forceinline__ void combine_waves(const KvAttnArgs &a, const float (*red)[D + 2],
                                              int64_t qi, int split, int tid)
{
    const float inf = __builtin_inff();
    if (tid < D) {
        float mx = red[0][0];
#pragma unroll
        for (int w = 1; w < ATT_WAVES; ++w)
            mx = fmaxf(mx, red[w][0]);
        float lt = 0.0f, ot = 0.0f;
        if (mx > -inf) {
#pragma unroll
            for (int w = 0; w < ATT_WAVES; ++w) {
                const float f = __expf(red[w][0] - mx);  // 0 for an empty wave
                lt = __builtin_fmaf(red[w][1], f, lt);
                ot = __builtin_fmaf(red[w][2 + tid], f, ot);
            }
        }
        if (a.splits == 1) {
            a.out[qi * D + tid] = f2h(ot / lt);
        } else {
            float *pp = a.part + (qi * a.splits + split) * (D + 2);
            if (tid == 0) {
                pp[0] = mx;
                pp[1] = lt;
            }
            pp[2 + tid] = ot;
        }
    }
}

template <int D>
__global__ __launch_bounds__(64 * ATT_WAVES) void k_kv_attn(KvAttnArgs a)
{
    constexpr int LPT = D / 32;       // lanes per token
    constexpr int TPW = 64 / LPT;     // tokens per wave load
    constexpr int LOGLPT = D == 64 ? 1 : D == 128 ? 2 : 3;
    __shared__ float red[ATT_WAVES][D + 2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t qi = blockIdx.x;
    const int split = blockIdx.y;
    const int64_t kvr = qi / a.rep;
    const int ds = (lane & (LPT - 1)) * 32;  // this lane's head-dim slice
    const int tl = lane >> LOGLPT;           // token within a load
    const int ng = D / a.G;
    const int gidx = ds / a.G;
    const int t_begin = split * a.chunk;
    const int t_end = min(a.seq_len, t_begin + a.chunk);

    float qv[32];
    float qsum = 0.0f;
    {
        const uint16_t *qr = a.q + qi * D + ds;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint4 raw = *reinterpret_cast<const uint4 *>(qr + 8 * p);
            const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                qv[8 * p + 2 * i] = h2f((uint16_t)(w[i] & 0xFFFFu));
                qv[8 * p + 2 * i + 1] = h2f((uint16_t)(w[i] >> 16));
            }
        }
#pragma unroll
        for (int e = 0; e < 32; ++e)
            qsum += qv[e];
    }

    float o[32];
#pragma unroll
    for (int e = 0; e < 32; ++e)
        o[e] = 0.0f;
    float m = -__builtin_inff(), l = 0.0f, zs = 0.0f;
    const int64_t rbase = kvr * a.s_max;
    const float inf = __builtin_inff();

    for (int base = t_begin + wave * TPW * ATT_U; base < t_end;
         base += ATT_WAVES * TPW * ATT_U) {
        uint4 kc[ATT_U], vc[ATT_U];
        float ksc[ATT_U], kze[ATT_U], vsc[ATT_U], vze[ATT_U];
        bool ok[ATT_U];
#pragma unroll
        for (int u = 0; u < ATT_U; ++u) {
            const int t = base + u * TPW + tl;
            ok[u] = t < t_end;
            const int64_t row = rbase + (ok[u] ? t : t_end - 1);
            kc[u] = *reinterpret_cast<const uint4 *>(a.kc + row * (D / 2) + ds / 2);
            vc[u] = *reinterpret_cast<const uint4 *>(a.vc + row * (D / 2) + ds / 2);
            ksc[u] = h2f(a.ks[row * ng + gidx]);
            kze[u] = h2f(a.kz[row * ng + gidx]);
            vsc[u] = h2f(a.vs[row * ng + gidx]);
            vze[u] = h2f(a.vz[row * ng + gidx]);
        }
        float sc[ATT_U];
        float tmax = -inf;
#pragma unroll
        for (int u = 0; u < ATT_U; ++u) {
            float s = __builtin_fmaf(ksc[u], dot_codes(kc[u], qv), kze[u] * qsum);
            static_for<LOGLPT>([&](auto J) { s = lane_sum<J>(s); });
            sc[u] = ok[u] ? s * a.sm_scale : -inf;
            tmax = fmaxf(tmax, sc[u]);
        }
        // the LPT lanes of a token hold the same score (their butterfly sums
        // add the same pairs), so the maximum runs over the other lane bits
        static_for<6>([&](auto J) {
            if constexpr (J >= LOGLPT)
                tmax = lane_max<J>(tmax);
        });
        const float mn = fmaxf(m, tmax);  // finite: every iteration has a token
        if (mn > m) {                     // uniform across the wave
            const float alpha = __expf(m - mn);
#pragma unroll
            for (int e = 0; e < 32; ++e)
                o[e] *= alpha;
            l *= alpha;
            zs *= alpha;
            m = mn;
        }
#pragma unroll
        for (int u = 0; u < ATT_U; ++u) {
            const float p = __expf(sc[u] - m);  // 0 for masked tokens
            l += p;
            zs = __builtin_fmaf(p, vze[u], zs);
            axpy_codes(vc[u], p * vsc[u], o);
        }
    }

    // sum over the lanes of a slice (one lane per token of a load)
    static_for<6>([&](auto J) {
        if (J >= LOGLPT) {
#pragma unroll
            for (int e = 0; e < 32; ++e)
                o[e] = lane_sum<J>(o[e]);
            l = lane_sum<J>(l);
            zs = lane_sum<J>(zs);
        }
    });
    if (tl == 0) {
#pragma unroll
        for (int e = 0; e < 32; ++e)
            red[wave][2 + ds + e] = o[e] + zs;
        if (ds == 0) {
            red[wave][0] = m;
            red[wave][1] = l;
        }
    }
    __syncthreads();
    combine_waves<D>(a, red, qi, split, tid);
}

// ---- head_dim 128 with one scale and zero per cached row: on the matrix
// cores.  A wave takes its tokens 16 at a time (lane l: token n = l % 16,
// lane group g = l / 16).
//
// Scores: v_mfma_f32_16x16x32_f16 with A = the query (every row the same)
// and B = the K codes as fp16 integers, contracting over head_dim in four
// 32-wide steps kc.  Lane l loads the 16 code bytes of elements
// 32 g .. 32 g + 31 of its token and supplies, at step kc, elements
// 32 g + 8 kc + s(j), s = 0, 4, 1, 5, 2, 6, 3, 7 (the order in which the
// nibble pairs come out); the query is laid out the same way.  Every output
// row is then the token's dot product, exact up to the binary32
// accumulation.
//
// Values: v_mfma_f32_16x16x16_f16 with A = the tokens' weights p_t vs_t
// rounded to fp16 (every row the same) and B = the V codes, contracting over
// the 16 tokens.  Lane l loads code bytes 4 n .. 4 n + 3 (elements
// 8 n .. 8 n + 7) of tokens 4 g .. 4 g + 3, and output column n of step
// dc = 0..7 accumulates element 8 n + dc.  The weights' fp16 rounding
// (relative 2^-11, like that of the fp16 output) is the only change from
// the vector kernel's arithmetic; the zero-point term sum_t p_t vz_t and
// the softmax sums stay in binary32.
//
// A code c becomes an fp16 integer by or-ing it into the significand of a
// 16-bit lane holding 1024 (where fp16 values are spaced by 1), giving
// 1024 + c, and subtracting 1024, both exact; one 32-bit and-or converts
// the two nibbles at bits 0-3 and 16-19.
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef _Float16 h2v __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

// The nibbles at bits 4-7 and 20-23 need no shift: or-ed into 0x5400 (64,
// spacing 1/16) they read 64 + c.  The and-or is one v_and_or_b32 on
// register operands (gfx9 VOP3 takes no literal, and the compiler otherwise
// splits it into an and and an or).
struct NibConst {
    uint32_t mlo, mhi, glo, ghi;  // masks and magic exponents, in registers
};

template <bool HI>
__device__ __forceinline__ h2v nib_pair(uint32_t w, const NibConst &k)
{
    uint32_t x;
    __asm__("v_and_or_b32 %0, %1, %2, %3"
            : "=v"(x)
            : "v"(w), "v"(HI ? k.mhi : k.mlo), "v"(HI ? k.ghi : k.glo));
    const _Float16 b = HI ? (_Float16)-64.0f : (_Float16)-1024.0f;
    const h2v off = {b, b};
    return __builtin_bit_cast(h2v, x) + off;
}

__device__ __forceinline__ _Float16 bits_h(uint32_t b)
{
    return __builtin_bit_cast(_Float16, (uint16_t)b);
}

constexpr int MFMA_U = 4;  // 16-token groups per wave per iteration

__global__ __launch_bounds__(64 * ATT_WAVES) void k_kv_attn_mfma(KvAttnArgs a)
{
    constexpr int D = 128;
    __shared__ float red[ATT_WAVES][D + 2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = lane & 15, g = lane >> 4;
    const int64_t qi = blockIdx.x;
    const int split = blockIdx.y;
    const int64_t kvr = qi / a.rep;
    const int t_begin = split * a.chunk;
    const int t_end = min(a.seq_len, t_begin + a.chunk);
    const float inf = __builtin_inff();

    // the query as the score steps' A operands, and its sum
    v8h qa[4];
    float qsum = 0.0f;
    {
        const uint4 *qr = reinterpret_cast<const uint4 *>(a.q + qi * D + 32 * g);
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
            const uint4 raw = qr[kc];  // elements 32 g + 8 kc .. + 7
            const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
            _Float16 e[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                e[2 * i] = bits_h(w[i] & 0xFFFFu);
                e[2 * i + 1] = bits_h(w[i] >> 16);
            }
            qa[kc] = v8h{e[0], e[4], e[1], e[5], e[2], e[6], e[3], e[7]};
#pragma unroll
            for (int i = 0; i < 8; ++i)
                qsum += (float)e[i];
        }
        qsum = lane_sum<4>(qsum);
        qsum = lane_sum<5>(qsum);
    }

    // running output: element 8 n + dc in orun[dc]; each iteration's value
    // products go to fresh accumulators (every output row the same, row 0
    // read), so the rescaling below touches 8 values in vector registers and
    // the matrix accumulators are never copied
    float orun[8];
#pragma unroll
    for (int dc = 0; dc < 8; ++dc)
        orun[dc] = 0.0f;
    float m = -inf, l = 0.0f, zs = 0.0f;
    const NibConst nk = {0x000F000Fu, 0x00F000F0u, 0x64006400u, 0x54005400u};
    // this cache row block's codes and constants: wave-uniform bases, 32-bit
    // offsets (s_max * 64 bytes < 2^32)
    const int64_t rbase = kvr * a.s_max;
    const uint8_t *kcb = a.kc + rbase * (D / 2), *vcb = a.vc + rbase * (D / 2);
    const uint16_t *ksb = a.ks + rbase, *kzb = a.kz + rbase, *vsb = a.vs + rbase, *vzb = a.vz + rbase;

    for (int base = t_begin + wave * 16 * MFMA_U; base < t_end;
         base += ATT_WAVES * 16 * MFMA_U) {
        uint4 kc[MFMA_U];
        uint32_t vw[MFMA_U][4];
        float ksc[MFMA_U], kze[MFMA_U], vsc[MFMA_U], vze[MFMA_U];
        bool ok[MFMA_U];
#pragma unroll
        for (int u = 0; u < MFMA_U; ++u) {
            const int t0 = base + 16 * u, t = t0 + n;
            ok[u] = t < t_end;
            const uint32_t row = (uint32_t)(ok[u] ? t : t_end - 1);
            kc[u] = *reinterpret_cast<const uint4 *>(kcb + (row * (D / 2) + 16 * g));
            ksc[u] = h2f(ksb[row]);
            kze[u] = h2f(kzb[row]);
            vsc[u] = h2f(vsb[row]);
            vze[u] = h2f(vzb[row]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int tj = t0 + 4 * g + j;
                const uint32_t rj = (uint32_t)(tj < t_end ? tj : t_end - 1);
                vw[u][j] = *reinterpret_cast<const uint32_t *>(vcb + (rj * (D / 2) + 4 * n));
            }
        }
        float sc[MFMA_U];
        float tmax = -inf;
#pragma unroll
        for (int u = 0; u < MFMA_U; ++u) {
            v4f acc = {0.0f, 0.0f, 0.0f, 0.0f};
            const uint32_t w4[4] = {kc[u].x, kc[u].y, kc[u].z, kc[u].w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t w8 = w4[k] >> 8;
                const h2v p0 = nib_pair<false>(w4[k], nk), p1 = nib_pair<true>(w4[k], nk);
                const h2v p2 = nib_pair<false>(w8, nk), p3 = nib_pair<true>(w8, nk);
                const v8h b = {p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
                acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa[k], b, acc, 0, 0, 0);
            }
            const float s = __builtin_fmaf(ksc[u], acc[0], kze[u] * qsum);
            sc[u] = ok[u] ? s * a.sm_scale : -inf;
            tmax = fmaxf(tmax, sc[u]);
        }
        // over the 16 tokens of a row (the four rows hold the same tokens)
        static_for<4>([&](auto J) { tmax = lane_max<J>(tmax); });
        const float mn = fmaxf(m, tmax);  // finite: every iteration has a token
        if (mn > m) {                     // uniform across the wave
            const float alpha = __expf(m - mn);
#pragma unroll
            for (int dc = 0; dc < 8; ++dc)
                orun[dc] *= alpha;
            l *= alpha;
            zs *= alpha;
            m = mn;
        }
        v4f o[8];
#pragma unroll
        for (int u = 0; u < MFMA_U; ++u) {
            const float p = __expf(sc[u] - m);  // 0 for masked tokens
            l += p;
            zs = __builtin_fmaf(p, vze[u], zs);
            const float wt = p * vsc[u];
            // A operand: the weights of tokens 4 g .. 4 g + 3 (lanes
            // 16 g + 4 g + j of this row)
            v4h av;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                av[j] = (_Float16)__shfl(wt, 20 * g + j);
#pragma unroll
            for (int bt = 0; bt < 4; ++bt) {
                // byte bt of tokens 4 g, 4 g + 1 (and + 2, + 3) in bytes 0, 2
                const uint32_t sel = (uint32_t)bt | 0x0C00u | ((uint32_t)(4 + bt) << 16) | 0x0C000000u;
                const uint32_t x01 = perm_b32(vw[u][1], vw[u][0], sel);
                const uint32_t x23 = perm_b32(vw[u][3], vw[u][2], sel);
                const h2v lo01 = nib_pair<false>(x01, nk), lo23 = nib_pair<false>(x23, nk);
                const h2v hi01 = nib_pair<true>(x01, nk), hi23 = nib_pair<true>(x23, nk);
                const v4h blo = {lo01[0], lo01[1], lo23[0], lo23[1]};
                const v4h bhi = {hi01[0], hi01[1], hi23[0], hi23[1]};
                const v4f z = {0.0f, 0.0f, 0.0f, 0.0f};
                o[2 * bt] = __builtin_amdgcn_mfma_f32_16x16x16f16(av, blo, u ? o[2 * bt] : z, 0, 0, 0);
                o[2 * bt + 1] =
                    __builtin_amdgcn_mfma_f32_16x16x16f16(av, bhi, u ? o[2 * bt + 1] : z, 0, 0, 0);
            }
        }
#pragma unroll
        for (int dc = 0; dc < 8; ++dc)
            orun[dc] += o[dc][0];
    }

    // sums over the 16 tokens of a row
    static_for<4>([&](auto J) {
        l = lane_sum<J>(l);
        zs = lane_sum<J>(zs);
    });
    if (g == 0) {
#pragma unroll
        for (int dc = 0; dc < 8; ++dc)
            red[wave][2 + 8 * n + dc] = orun[dc] + zs;
        if (n == 0) {
            red[wave][0] = m;
            red[wave][1] = l;
        }
    }
    __syncthreads();
    combine_waves<D>(a, red, qi, split, tid);
}

// out[qi][d] from the splits' (max, sum, o): one block of D threads per row.
template <int D>
__global__ __launch_bounds__(D) void k_kv_attn_combine(KvAttnArgs a)
{
    const int64_t qi = blockIdx.x;
    const int d = threadIdx.x;
    const float *pp = a.part + qi * a.splits * (D + 2);
    float mx = -__builtin_inff();
    for (int s = 0; s < a.splits; ++s)
        mx = fmaxf(mx, pp[s * (D + 2)]);
    float lt = 0.0f, ot = 0.0f;
    for (int s = 0; s < a.splits; ++s) {
        const float ms = pp[s * (D + 2)];
        if (ms == -__builtin_inff())
            continue;  // an empty chunk
        const float f = __expf(ms - mx);
        lt = __builtin_fmaf(pp[s * (D + 2) + 1], f, lt);
        ot = __builtin_fmaf(pp[s * (D + 2) + 2 + d], f, ot);
    }
    a.out[qi * D + d] = f2h(ot / lt);
}

template <int D>
hipError_t go_attn(const KvAttnArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_kv_attn<D>, dim3((unsigned)a.nq, (unsigned)a.splits),
                       dim3(64 * ATT_WAVES), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits == 1)
        return e;
    hipLaunchKernelGGL(k_kv_attn_combine<D>, dim3((unsigned)a.nq), dim3(D), 0, s, a);
    return hipGetLastError();
}

hipError_t go_attn_mfma(const KvAttnArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_kv_attn_mfma, dim3((unsigned)a.nq, (unsigned)a.splits),
                       dim3(64 * ATT_WAVES), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits == 1)
        return e;
    hipLaunchKernelGGL(k_kv_attn_combine<128>, dim3((unsigned)a.nq), dim3(128), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_attention(const KvAttnArgs &a, hipStream_t s)
{
    if (a.nq == 0)
        return hipSuccess;
    switch (a.D) {
    case 64: return go_attn<64>(a, s);
    case 128:
        if (a.G == 128)
            return go_attn_mfma(a, s);
        return go_attn<128>(a, s);
    case 256: return go_attn<256>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace quarot
