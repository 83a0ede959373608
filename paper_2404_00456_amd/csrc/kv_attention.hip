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
// lane's 32 elements share one scale and zero.
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
    // combine the waves (thread d < D owns output element d)
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

}  // namespace

hipError_t launch_kv_attention(const KvAttnArgs &a, hipStream_t s)
{
    if (a.nq == 0)
        return hipSuccess;
    switch (a.D) {
    case 64: return go_attn<64>(a, s);
    case 128: return go_attn<128>(a, s);
    case 256: return go_attn<256>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace quarot
