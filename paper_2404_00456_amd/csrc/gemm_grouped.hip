// Group-wise W4A4 GEMM (§5.3 group-size ablation: a scale per group of
// 64, 128 or 256 input channels for activations and weights), for gfx950.
//
//   acc_g[m][n] = sum over k in group g of qx[m][k] qw[n][k]     (int32, exact)
//   y[m][n]     = RN16(((+0 + t_0) + t_1) + ...),
//   t_g         = RN(RN(f32(acc_g) sx[g][m]) sw[g][n])            (binary32)
//
// Operand widening, tile order and LDS DMA as in the per-token kernel.
#include "gemm_common.hpp"

namespace quarot {
namespace {

using namespace gemm;

// ------------------------------------------------------------------------
// Group-wise W4A4 (a scale per group of GS = 64, 128 or 256 input channels
// for activations and weights).  A k-step covers KS = max(GS, 128) k; the
// MFMA substeps of one group accumulate its integer product in a temporary
// (256 acc_g, exact), which is dequantized at once,
// t = RN(RN(f32(acc_g) sx[g][m]) sw[g][n]), and added to binary32 output
// accumulators in group order.  The binary32 accumulators live in VGPRs
// next to the MFMA temporaries, so a wave covers 64 x 64 (block 256 x 128,
// waves 4 x 2; the per-token kernel's waves cover 128 x 64).  Scales are
// group-major (sx [K/GS, M], sw [K/GS, N]) and staged in LDS with the
// operands of their k-step.  This kernel takes any M and N; the ring kernel
// below takes M and N multiples of 8.
constexpr int GBN = 128;  // W rows per block

// Integer to binary32 without a conversion instruction: an MFMA temporary
// started at kMagic (the bits of M = 1.5 * 2^23) instead of 0 ends as the
// bits of M + 256 acc_g, since |256 acc_g| <= 2^22 keeps the sum in
// [2^23, 2^24], where the float spacing is 1.  Hence (bits as float) - M is
// f32(256 acc_g) exactly, and with sxc = sx / 256 (an fp16 significand, 11
// bits) the product M * sxc has at most 12 significant bits and is exact,
// so fma(bits as float, sxc, -M * sxc) = RN(f32(acc_g) sx) in one step.
constexpr int kMagic = 0x4B400000;
constexpr float kMagicF = 0x1.8p23f;

template <int GS>
struct GroupTile {
    static constexpr int KS = GS < 128 ? 128 : GS;  // k per k-step
    static constexpr int SUB = KS / 64;             // MFMA substeps per k-step
    static constexpr int GSUB = GS / 64;            // substeps per group
    static constexpr int GPS = KS / GS;             // groups per k-step
    static constexpr int ROWB = KS / 2;             // packed bytes per row per k-step
    static constexpr int PITCH = ROWB + 16;         // LDS row pitch
    static constexpr int TILE = (BM + GBN) * PITCH;
    static constexpr int SCB = GPS * (BM + GBN) * 2;  // scale bytes: sx [GPS][BM], sw [GPS][GBN]
    static constexpr int STAGE = TILE + SCB;
    static constexpr int NSC = SCB / 16;              // 16-byte scale chunks per stage
    static constexpr int LDS = 2 * STAGE;
    static constexpr int CPR = ROWB / 16;           // 16-byte chunks per row
    static constexpr int NLX = BM * CPR / THREADS;  // X chunks per thread
    static constexpr int NLW = GBN * CPR / THREADS; // W chunks per thread
    static constexpr bool CACHE_W = GS <= 128;      // W fragments kept across j
    static constexpr bool FLOAT_SW = GPS == 1;      // sw held converted, else packed
};

template <int GS>
__global__ __launch_bounds__(THREADS, 1) void k_gemm_w4a4_grouped(GemmArgs a)
{
    using T = GroupTile<GS>;
    extern __shared__ __align__(16) uint8_t lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;  // 64-row x 64-column wave tiles
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + BM - 1) / BM, TN = (N + GBN - 1) / GBN;
    int tm, tn;
    tile_of(blockIdx.x, gridDim.x, TM, TN, tm, tn);
    const int m0 = tm * BM, n0 = tn * GBN;
    const int64_t ldk = K / 2;
    const int KT = K / T::KS;

    // global -> LDS: 16-byte chunk id = tid + 512 i, CPR chunks per row
    const uint8_t *gx[T::NLX];
    const uint8_t *gw[T::NLW];
    int xrow[T::NLX], xcol[T::NLX], wrow[T::NLW], wcol[T::NLW];
#pragma unroll
    for (int i = 0; i < T::NLX; ++i) {
        const int id = tid + THREADS * i;
        xrow[i] = id / T::CPR;
        xcol[i] = id % T::CPR;
        gx[i] = a.xq + (int64_t)min(m0 + xrow[i], M - 1) * ldk + xcol[i] * 16;
    }
#pragma unroll
    for (int i = 0; i < T::NLW; ++i) {
        const int id = tid + THREADS * i;
        wrow[i] = id / T::CPR;
        wcol[i] = id % T::CPR;
        gw[i] = a.wq + (int64_t)min(n0 + wrow[i], N - 1) * ldk + wcol[i] * 16;
    }

    const int orow = lane & 15;
    const int obyte = (lane >> 4) * 8;
    const bool nvec = (N & 3) == 0;

    // scales: thread tid < NSC fetches 8 consecutive fp16 of one group's
    // sx (chunks 0..32 GPS - 1) or sw (the rest) of the next k-step
    constexpr int XCH = BM / 8, WCH = GBN / 8;  // chunks per group
    const bool sc_ld = tid < T::NSC;
    const int sc_g2 = tid < T::GPS * XCH ? tid / XCH : (tid - T::GPS * XCH) / WCH;
    const bool sc_x = tid < T::GPS * XCH;
    const int sc_c = sc_x ? tid % XCH : (tid - T::GPS * XCH) % WCH;
    const int sc_lim = sc_x ? M : N;                    // rows of the scale vector
    const int sc_e0 = (sc_x ? m0 : n0) + sc_c * 8;      // first element
    const bool sc_vec = ((sc_x ? M : N) & 7) == 0 && sc_e0 + 7 < sc_lim;
    const int sc_lds = T::TILE + (sc_x ? sc_g2 * BM + sc_c * 8
                                       : T::GPS * BM + sc_g2 * GBN + sc_c * 8) * 2;

    uint4 px[T::NLX], pw[T::NLW], psc;
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < T::NLX; ++i)
            px[i] = *reinterpret_cast<const uint4 *>(gx[i] + (int64_t)kt * T::ROWB);
#pragma unroll
        for (int i = 0; i < T::NLW; ++i)
            pw[i] = *reinterpret_cast<const uint4 *>(gw[i] + (int64_t)kt * T::ROWB);
        if (sc_ld) {
            const int64_t g = (int64_t)kt * T::GPS + sc_g2;
            const uint16_t *v = (sc_x ? a.sx : a.sw) + g * sc_lim;
            if (sc_vec) {
                psc = *reinterpret_cast<const uint4 *>(v + sc_e0);
            } else {
                uint32_t h[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    h[e] = v[min(sc_e0 + e, sc_lim - 1)];
                psc = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                                 h[6] | (h[7] << 16));
            }
        }
    };
    auto lstore = [&](int stage) {
        uint8_t *base = lds + stage * T::STAGE;
#pragma unroll
        for (int i = 0; i < T::NLX; ++i)
            *reinterpret_cast<uint4 *>(base + xrow[i] * T::PITCH + xcol[i] * 16) = px[i];
#pragma unroll
        for (int i = 0; i < T::NLW; ++i)
            *reinterpret_cast<uint4 *>(base + (BM + wrow[i]) * T::PITCH + wcol[i] * 16) = pw[i];
        if (sc_ld)
            *reinterpret_cast<uint4 *>(base + sc_lds) = psc;
    };
    // this k-step's scales from LDS: sx divided by 256; sw converted (one
    // group per k-step) or kept packed and converted at use (two groups)
    float sxc[T::GPS][4], swc[T::FLOAT_SW ? 4 : 1][4];
    uint2 swp[T::FLOAT_SW ? 1 : T::GPS][4];
    auto scales = [&](const uint8_t *sb) {
        const uint16_t *lsx = reinterpret_cast<const uint16_t *>(sb + T::TILE);
        const uint16_t *lsw = lsx + T::GPS * BM;
#pragma unroll
        for (int g2 = 0; g2 < T::GPS; ++g2) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                sxc[g2][j] = h2f(lsx[g2 * BM + wm * 64 + j * 16 + orow]) * 0x1p-8f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint2 w2 = *reinterpret_cast<const uint2 *>(
                    lsw + g2 * GBN + wn * 64 + i * 16 + (lane >> 4) * 4);
                if constexpr (T::FLOAT_SW) {
                    swc[i][0] = h2f((uint16_t)w2.x);
                    swc[i][1] = h2f((uint16_t)(w2.x >> 16));
                    swc[i][2] = h2f((uint16_t)w2.y);
                    swc[i][3] = h2f((uint16_t)(w2.y >> 16));
                } else {
                    swp[g2][i] = w2;
                }
            }
        }
    };
    auto swv = [&](int g2, int i, int r) {
        if constexpr (T::FLOAT_SW)
            return swc[i][r];
        else {
            const uint32_t w = r < 2 ? swp[g2][i].x : swp[g2][i].y;
            return h2f((uint16_t)(w >> (16 * (r & 1))));
        }
    };

    float yacc[4][4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                yacc[i][j][r] = 0.0f;

    gload(0);
    lstore(0);
    __syncthreads();

    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT)
            gload(kt + 1);
        const uint8_t *sb = lds + cur * T::STAGE;
        scales(sb);
        auto wfrag = [&](int kk, int i) {
            return widen(*reinterpret_cast<const uint2 *>(
                sb + (BM + wn * 64 + i * 16 + orow) * T::PITCH + kk * 32 + obyte));
        };
        v4i aq[T::CACHE_W ? T::SUB : 1][4];
        if constexpr (T::CACHE_W) {
#pragma unroll
            for (int kk = 0; kk < T::SUB; ++kk)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    aq[kk][i] = wfrag(kk, i);
        }
        // units u = (j, g2): the MFMAs of unit u + 1 are issued before the
        // dequant of unit u, and nothing moves across units, so two sets of
        // temporaries are live at a time
        constexpr int U = 4 * T::GPS;
        auto mfma_unit = [&](auto UI, v4i(&t)[4]) {
            constexpr int j = decltype(UI)::value / T::GPS, g2 = decltype(UI)::value % T::GPS;
            if constexpr (!T::CACHE_W)  // W fragments are read again per unit, not kept
                __asm__ volatile("" ::: "memory");
            const uint8_t *p = sb + (wm * 64 + j * 16 + orow) * T::PITCH + obyte;
#pragma unroll
            for (int s2 = 0; s2 < T::GSUB; ++s2) {
                const int kk = g2 * T::GSUB + s2;
                const v4i bq = widen(*reinterpret_cast<const uint2 *>(p + kk * 32));
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v4i w;
                    if constexpr (T::CACHE_W)
                        w = aq[kk][i];
                    else
                        w = wfrag(kk, i);
                    t[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                        w, bq, s2 == 0 ? v4i{0, 0, 0, 0} : t[i], 0, 0, 0);
                }
            }
        };
        // f32(256 acc_g) (sx / 256) is RN(f32(acc_g) sx): the same real, no
        // overflow or underflow; then * sw, then the add
        auto dequant_unit = [&](auto UI, const v4i(&t)[4]) {
            constexpr int j = decltype(UI)::value / T::GPS, g2 = decltype(UI)::value % T::GPS;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float u = ((float)t[i][r] * sxc[g2][j]) * swv(g2, i, r);
                    yacc[i][j][r] = yacc[i][j][r] + u;
                    // pinned here: otherwise the dequant sinks below the
                    // later units' MFMAs and all their temporaries stay live
                    __asm__ volatile("" : "+v"(yacc[i][j][r]));
                }
        };
        v4i ta[4], tb[4];
        mfma_unit(std::integral_constant<int, 0>{}, ta);
        static_for<U>([&](auto UI) {
            constexpr int u = decltype(UI)::value;
            if constexpr (u + 1 < U)
                mfma_unit(std::integral_constant<int, u + 1>{}, (u & 1) ? ta : tb);
            __builtin_amdgcn_sched_barrier(0);
            dequant_unit(UI, (u & 1) ? tb : ta);
            __builtin_amdgcn_sched_barrier(0);
        });
        if (kt + 1 < KT)
            lstore(cur ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int nb = n0 + wn * 64 + i * 16 + (lane >> 4) * 4;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + j * 16 + orow;
            if (m >= M)
                continue;
            uint16_t hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
                hv[r] = f2h(yacc[i][j][r]);
            uint16_t *yrow = a.y + (int64_t)m * N;
            if (nvec && nb + 3 < N) {
                uint2 pk;
                pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                *reinterpret_cast<uint2 *>(yrow + nb) = pk;
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (nb + r < N)
                        yrow[nb + r] = hv[r];
            }
        }
    }
}

// ------------------------------------------------------------------------
// Group-wise W4A4, persistent with an LDS-DMA ring (M and N multiples of 8).
// The group arithmetic is that of k_gemm_w4a4_grouped above (one integer
// temporary per group and wave slice, dequantized at once and added to
// binary32 accumulators in group order); the operand path is that of the
// per-token kernel's main path: HBM -> LDS by global_load_lds, RS stages, RS - 1 k-steps in
// flight, one barrier per k-step, the ring running on across the tiles a
// block walks.  A k-step (KS = max(GS, 128) k) stages 256 X rows and 128 W
// rows of KS / 2 bytes, unpadded, with 16-byte unit c of row r stored at
// c ^ swz(r) (swz = (r >> 1) & 3 for 64-byte rows, r & 7 for 128-byte
// rows), and the k-step's group scales: every wave adds one 4-byte-per-lane
// DMA (sx halves, sw, or a dummy slot) so that all waves count the same
// loads.
//
// k assignment (identical for both operands, so dot products are unchanged
// and each MFMA substep stays within one group):
//  * 128-byte rows (GS 256): lane group q = lane / 16 reads units q and
//    q + 4; substeps 0, 1 take the halves of unit q, 2, 3 those of q + 4.
//  * 64-byte rows, GS 128: unit q; substeps 0, 1 its two halves.
//  * 64-byte rows, GS 64: substep s (= group s of the step) takes the
//    8 bytes at 32 s + 8 q, so substep s covers exactly bytes [32 s, 32 s + 32).
template <int GS>
struct GroupRing {
    static constexpr int KS = GS < 128 ? 128 : GS;
    static constexpr int ROWB = KS / 2;                // packed bytes per row per k-step
    static constexpr int UNITS = ROWB / 16;            // 16-byte units per row
    static constexpr int SUB = KS / 64;                // MFMA substeps per k-step
    static constexpr int GSUB = GS / 64;               // substeps per group
    static constexpr int GPS = KS / GS;                // groups per k-step
    static constexpr int RS = GS == 256 ? 3 : 4;       // ring stages
    static constexpr int OPB = (BM + GBN) * ROWB;      // operand bytes per stage
    static constexpr int SCL = 8 * 256;                // scale slots: one 256-byte slot per wave
    static constexpr int STAGE = OPB + SCL;
    static constexpr int LDS = RS * STAGE;
    static constexpr int RPC = 1024 / ROWB;            // rows per 1 KB DMA
    static constexpr int DPW = OPB / 1024 / 8;         // operand DMAs per wave per k-step
    static constexpr int D = DPW + 1;                  // all DMAs per wave per k-step
    static constexpr int NR = GS == 128 ? 1 : 2;       // LDS reads per slice per k-step
};

template <int ROWB>
__device__ __forceinline__ int ring_swz(int r)
{
    return ROWB == 64 ? (r >> 1) & 3 : r & 7;
}

template <int GS>
__global__ __launch_bounds__(THREADS, 1) void k_gemm_w4a4_grouped_ring(GemmArgs a)
{
    using C = GroupRing<GS>;
    extern __shared__ __align__(16) uint8_t lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;  // 64 x 64 wave tiles
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + BM - 1) / BM, TN = (N + GBN - 1) / GBN;
    const int T = TM * TN;
    const int G = gridDim.x, b = blockIdx.x;
    const int64_t ldk = K / 2;
    const int KT = K / C::KS;

    const bool xcd = (G % 8 == 0) && (T % 8 == 0) && G <= T;
    auto tile_pos = [&](int it) -> int {
        if (xcd) {
            const int per_x = T / 8, gx = G / 8;
            const int r = (b >> 3) + it * gx;
            return r < per_x ? (b & 7) * per_x + r : -1;
        }
        const int t = b + it * G;
        return t < T ? t : -1;
    };
    auto tile_mn = [&](int t, int &m0, int &n0) {
        const int gsize = GM * TN;
        const int g = t / gsize;
        const int first = g * GM;
        const int gm = min(TM - first, GM);
        const int r = t - g * gsize;
        m0 = (first + r % gm) * BM;
        n0 = (r / gm) * GBN;
    };

    // operand DMA i of wave w: 1 KB chunk c = w + 8 i of the stage (X rows
    // 0..255 first, then W rows); lane l fills LDS unit l % UNITS of row
    // c * RPC + l / UNITS and so fetches global unit (l % UNITS) ^ swz(row)
    int drow[C::DPW], dunit[C::DPW];
#pragma unroll
    for (int i = 0; i < C::DPW; ++i) {
        const int r = (wave + 8 * i) * C::RPC + lane / C::UNITS;
        drow[i] = r;
        dunit[i] = (lane % C::UNITS) ^ ring_swz<C::ROWB>(r);
    }
    // SGPR-base form: a per-lane 32-bit offset inside the tile's rows (rows
    // past the matrix edge clamped), fixed per tile, and a wave-uniform base
    // advanced by one k-step per issue.  Whether DMA i moves X or W rows is
    // uniform per wave (a chunk never straddles row BM).
    bool dx[C::DPW];
    int dsts[C::DPW];
#pragma unroll
    for (int i = 0; i < C::DPW; ++i) {
        dx[i] = __builtin_amdgcn_readfirstlane((wave + 8 * i) * C::RPC) < BM;
        dsts[i] = __builtin_amdgcn_readfirstlane((wave + 8 * i) * 1024);
    }
    auto voffG = [&](int i, int m0, int n0) -> uint32_t {
        const int r = dx[i] ? min(drow[i], M - 1 - m0) : min(drow[i] - BM, N - 1 - n0);
        return (uint32_t)(r * (int)ldk + dunit[i] * 16);
    };
    auto baseG = [&](int i, int m0, int n0, int sk) -> const uint8_t * {
        return (dx[i] ? a.xq + (int64_t)m0 * ldk : a.wq + (int64_t)n0 * ldk) +
               (int64_t)sk * C::ROWB;
    };
    // scale DMA of wave w: slot w of the stage's scale area.  Slots 0..2GPS-1
    // hold sx of group g2 = w / 2 (128 rows each), slots 2GPS..3GPS-1 sw of
    // group w - 2GPS; the other waves fetch slot 0's source into their own
    // slot (never read).  2 fp16 per lane, element index clamped to an even
    // one inside the vector.
    const int sw_slot = wave - 2 * C::GPS;
    const bool sc_x = wave < 2 * C::GPS || sw_slot >= C::GPS;
    const int sc_g2 = wave < 2 * C::GPS ? wave >> 1 : (sw_slot < C::GPS ? sw_slot : 0);
    const int sc_half = wave < 2 * C::GPS ? wave & 1 : 0;
    auto scale_src = [&](int m0, int n0, int kt) -> const uint16_t * {
        const int64_t g = (int64_t)kt * C::GPS + sc_g2;
        if (sc_x)
            return a.sx + g * M + min(m0 + 128 * sc_half + 2 * lane, M - 2);
        return a.sw + g * N + min(n0 + 2 * lane, N - 2);
    };

    const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_void *)lds;
    uint32_t vo[C::DPW];
    const uint8_t *bcur[C::DPW];
    auto issue = [&](const uint8_t *const (&base)[C::DPW], const uint16_t *ssrc, int stage) {
        const uint32_t sbase = lds_base + stage * C::STAGE;
#pragma unroll
        for (int i = 0; i < C::DPW; ++i)
            dma16s(vo[i], base[i], sbase + dsts[i]);
        dma4(ssrc, __builtin_amdgcn_readfirstlane(sbase + C::OPB + wave * 256));
    };

    const int orow = lane & 15, q = lane >> 4;
    // operand reads: byte offset of read k of this lane in row r (see the
    // k assignment above; units stored swizzled)
    auto row_off = [&](int r, int k) -> int {
        const int byte = GS == 64 ? 32 * k + 8 * q : 16 * (q + 4 * k);
        const int u = byte >> 4;
        return r * C::ROWB + ((u ^ ring_swz<C::ROWB>(r)) << 4) + (byte & 15);
    };
    // X slices j (MFMA B operand), W slices i (A operand)
    int xoff[4][C::NR], woff[4][C::NR];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int k = 0; k < C::NR; ++k) {
            xoff[j][k] = row_off(wm * 64 + j * 16 + orow, k);
            woff[j][k] = row_off(BM + wn * 64 + j * 16 + orow, k);
        }

    int t = tile_pos(0);
    if (t < 0)
        return;
    int m0, n0;
    tile_mn(t, m0, n0);
#pragma unroll
    for (int i = 0; i < C::DPW; ++i)
        vo[i] = voffG(i, m0, n0);
    // global step g of this block lives in stage g % RS
    int g = 0;
#pragma unroll
    for (int s = 0; s < C::RS - 1; ++s) {
        const uint8_t *b0[C::DPW];
#pragma unroll
        for (int i = 0; i < C::DPW; ++i)
            b0[i] = baseG(i, m0, n0, min(s, KT - 1));
        issue(b0, scale_src(m0, n0, min(s, KT - 1)), s);
    }
#pragma unroll
    for (int i = 0; i < C::DPW; ++i)
        bcur[i] = baseG(i, m0, n0, C::RS - 1);
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((C::RS - 2) * C::D, 15));
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");

    for (int it = 0; t >= 0; ++it) {
        const int tn_ = tile_pos(it + 1);
        int m1 = 0, n1 = 0;
        if (tn_ >= 0)
            tile_mn(tn_, m1, n1);

        float yacc[4][4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    yacc[i][j][r] = 0.0f;

        for (int kt = 0; kt < KT; ++kt, ++g) {
            // DMA of global step g + RS - 1 into the stage read in step
            // g - 1 (every wave finished those reads before the last
            // barrier): this tile's step kt + RS - 1, else the next tile's,
            // else (no next tile) a harmless re-fetch
            {
                const bool here = kt + C::RS - 1 < KT;
                const bool cur = here || tn_ < 0;
                const int sk = here ? kt + C::RS - 1 : (tn_ >= 0 ? kt + C::RS - 1 - KT : KT - 1);
                const int stage = (g + C::RS - 1) % C::RS;
                if (here || tn_ >= 0) {
                    // the next tile's bases and lane offsets replace this
                    // tile's when the first of its DMAs is issued
                    if (kt + C::RS - 1 == KT) {
#pragma unroll
                        for (int i = 0; i < C::DPW; ++i) {
                            vo[i] = voffG(i, m1, n1);
                            bcur[i] = baseG(i, m1, n1, 0);
                        }
                    }
                    issue(bcur, scale_src(cur ? m0 : m1, cur ? n0 : n1, sk), stage);
#pragma unroll
                    for (int i = 0; i < C::DPW; ++i)
                        bcur[i] += C::ROWB;
                } else {
                    const uint8_t *b0[C::DPW];
#pragma unroll
                    for (int i = 0; i < C::DPW; ++i)
                        b0[i] = baseG(i, m0, n0, KT - 1);
                    issue(b0, scale_src(m0, n0, KT - 1), stage);
                }
            }
            const uint8_t *sb = lds + (g % C::RS) * C::STAGE;
            // operands of this step
            uint4 xr[4][C::NR], wr[4][C::NR];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int k = 0; k < C::NR; ++k) {
                    if constexpr (GS == 64) {
                        const uint2 xv = *reinterpret_cast<const uint2 *>(sb + xoff[j][k]);
                        const uint2 wv = *reinterpret_cast<const uint2 *>(sb + woff[j][k]);
                        xr[j][k] = make_uint4(xv.x, xv.y, 0, 0);
                        wr[j][k] = make_uint4(wv.x, wv.y, 0, 0);
                    } else {
                        xr[j][k] = *reinterpret_cast<const uint4 *>(sb + xoff[j][k]);
                        if constexpr (GS != 256)  // GS 256: read per unit (registers)
                            wr[j][k] = *reinterpret_cast<const uint4 *>(sb + woff[j][k]);
                    }
                }
            // 8 bytes of substep s from the reads
            auto half8 = [&](const uint4 (&v)[C::NR], int s) -> uint2 {
                if constexpr (GS == 64)
                    return make_uint2(v[s].x, v[s].y);
                else {
                    const uint4 u = v[s >> 1];
                    return (s & 1) ? make_uint2(u.z, u.w) : make_uint2(u.x, u.y);
                }
            };
            // this step's scales: sx / 256, sw converted (one group per
            // step) or packed and converted at use (two groups)
            const uint16_t *lsc = reinterpret_cast<const uint16_t *>(sb + C::OPB);
            float sxc[C::GPS][4], nsxc[C::GPS][4];
            float swc[C::GPS == 1 ? 4 : 1][4];
            uint2 swp[C::GPS == 1 ? 1 : C::GPS][4];
#pragma unroll
            for (int g2 = 0; g2 < C::GPS; ++g2) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    sxc[g2][j] = h2f(lsc[256 * g2 + wm * 64 + j * 16 + orow]) * 0x1p-8f;
                    nsxc[g2][j] = -(kMagicF * sxc[g2][j]);  // exact: 12 significant bits
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint2 w2 = *reinterpret_cast<const uint2 *>(
                        lsc + 256 * C::GPS + 128 * g2 + wn * 64 + i * 16 + q * 4);
                    if constexpr (C::GPS == 1) {
                        swc[i][0] = h2f((uint16_t)w2.x);
                        swc[i][1] = h2f((uint16_t)(w2.x >> 16));
                        swc[i][2] = h2f((uint16_t)w2.y);
                        swc[i][3] = h2f((uint16_t)(w2.y >> 16));
                    } else {
                        swp[g2][i] = w2;
                    }
                }
            }
            auto swv = [&](int g2, int i, int r) {
                if constexpr (C::GPS == 1)
                    return swc[i][r];
                else {
                    const uint32_t w = r < 2 ? swp[g2][i].x : swp[g2][i].y;
                    return h2f((uint16_t)(w >> (16 * (r & 1))));
                }
            };

            constexpr int U = 4 * C::GPS;
            auto mfma_unit = [&](auto UI, v4i(&tt)[4]) {
                constexpr int j = decltype(UI)::value / C::GPS, g2 = decltype(UI)::value % C::GPS;
                if constexpr (GS == 256)  // W fragments read again per unit, not kept
                    __asm__ volatile("" ::: "memory");
#pragma unroll
                for (int s2 = 0; s2 < C::GSUB; ++s2) {
                    const int sub = g2 * C::GSUB + s2;
                    const v4i bq = widen(half8(xr[j], sub));
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        uint2 w8;
                        if constexpr (GS == 256)
                            w8 = *reinterpret_cast<const uint2 *>(sb + woff[i][sub >> 1] +
                                                                  (sub & 1) * 8);
                        else
                            w8 = half8(wr[i], sub);
                        tt[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                            widen(w8), bq, s2 == 0 ? v4i{kMagic, kMagic, kMagic, kMagic} : tt[i],
                            0, 0, 0);
                    }
                }
            };
            // the temporaries hold M + 256 acc_g as binary32 bits (see
            // kMagic): fma(that, sx / 256, -M sx / 256) = RN(f32(acc_g) sx)
            auto dequant_unit = [&](auto UI, const v4i(&tt)[4]) {
                constexpr int j = decltype(UI)::value / C::GPS, g2 = decltype(UI)::value % C::GPS;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int bits = tt[i][r];  // (a vector element is not bit_cast directly)
                        const float v = __int_as_float(bits);
                        const float u = __builtin_fmaf(v, sxc[g2][j], nsxc[g2][j]) * swv(g2, i, r);
                        yacc[i][j][r] = yacc[i][j][r] + u;
                        __asm__ volatile("" : "+v"(yacc[i][j][r]));
                    }
            };
            v4i ta[4], tb[4];
            mfma_unit(std::integral_constant<int, 0>{}, ta);
            static_for<U>([&](auto UI) {
                constexpr int u = decltype(UI)::value;
                if constexpr (u + 1 < U)
                    mfma_unit(std::integral_constant<int, u + 1>{}, (u & 1) ? ta : tb);
                dequant_unit(UI, (u & 1) ? tb : ta);
                // the next unit's MFMAs spread among this unit's dequant, so
                // the matrix core works while the VALU does
                if constexpr (u + 1 < U) {
                    constexpr int NM = 4 * C::GSUB;
#pragma unroll
                    for (int k = 0; k < NM; ++k) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 56 / NM, 0);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            });

            // step g + 1 landed for this wave's DMAs (RS - 2 later steps may
            // stay in flight; loads complete in order, and stores issued in
            // between only make the wait longer), every LDS read of stage
            // g % RS done; then for every wave
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm((C::RS - 2) * C::D, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
        }

        // epilogue: lane holds n = nb + r (r < 4) of m = mb + orow per slice
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + j * 16 + orow;
            if (m >= M)
                continue;
            uint16_t *yrow = a.y + (int64_t)m * N;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int nb = n0 + wn * 64 + i * 16 + q * 4;
                if (nb >= N)
                    continue;  // N is a multiple of 8: a quad is all in or all out
                const h2 lo = __builtin_convertvector((f2){yacc[i][j][0], yacc[i][j][1]}, h2);
                const h2 hi = __builtin_convertvector((f2){yacc[i][j][2], yacc[i][j][3]}, h2);
                uint2 pk;
                pk.x = __builtin_bit_cast(uint32_t, lo);
                pk.y = __builtin_bit_cast(uint32_t, hi);
                *reinterpret_cast<uint2 *>(yrow + nb) = pk;
            }
        }

        t = tn_;
        m0 = m1;
        n0 = n1;
    }
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));  // no DMA may outlive the block's LDS
}


// RN(a h) for a binary32 a and an fp16 h as fma(a, h, +0): one
// v_fma_mix_f32 that takes h from its half of a register, no conversion.
// It differs from the plain product only where that is -0, which it
// returns as +0.  In the dequant below a zero first product makes the
// second one a zero as well, and the second is added into a sum that
// starts at +0; such a sum never becomes -0 (x + y is -0 in
// round-to-nearest only when both are -0), so adding +0 instead of -0
// leaves it as it is.
__device__ __forceinline__ float mul_h(float a, _Float16 h)
{
    return __builtin_fmaf(a, (float)h, 0.0f);
}

// ------------------------------------------------------------------------
// Group-wise product on e3m2 operands (the tiled layout of k_pack_e3m2),
// groups of 128 or 256.  A k-step is one 128-k block of the layout and a
// group is GS / 128 consecutive k-steps.  One v_mfma_f32_16x16x128_f8f6f4
// per 16 x 16 slice pair and k-step accumulates the group's products in a
// binary32 temporary; every product of two codes is an integer of
// magnitude <= 64 and |acc_g| <= 64 GS < 2^24, so the temporary is
// f32(acc_g) exactly, and the dequant is two multiplies and an add per
// output: t = RN(RN(tmp sx[g][m]) sw[g][n]), y_acc = y_acc + t.  No
// widening, and half the MFMAs of the int4 path.
//
// Block tile 256 (m) x 128 (n), eight waves of 64 x 64 as in the int4 ring
// kernel; a ring of RS stages, each holding the 64-byte heads of the 384
// stage rows (X rows, then W rows), their 32-byte tails (same order), and
// the step's group scales: sx in two 256-byte slots, sw in one, a fourth
// slot for a dummy load.  DMAs of wave w per k-step (1 KB each except the
// 256-byte scale loads; every instruction reads consecutive bytes):
//   0, 1  X heads of stage rows 16 w .. + 15 and 128 + 16 w .. + 15
//   2     W heads of W rows 16 w .. + 15
//   3     X tails of stage rows 32 w .. + 31
//   4     waves 0-3: W tails of W rows 32 w .. + 31; waves 4, 5: sx slots
//         0, 1; wave 6: sw; wave 7: sw again into the dummy slot
// so that every wave counts the same D = 5 loads in its vmcnt waits.
template <int GS>
struct GroupRing6 {
    static constexpr int GST = GS / 128;           // k-steps per group
    static constexpr int ROWS = BM + GBN;          // stage rows
    static constexpr int HEADS = ROWS * 64;        // offset of the tails
    static constexpr int SCL = HEADS + ROWS * 32;  // offset of the scale slots
    static constexpr int STAGE = SCL + 4 * 256;
    static constexpr int RS = 4;                   // ring stages
    static constexpr int LDS = RS * STAGE;
    static constexpr int D = 5;                    // loads per wave per k-step
};

template <int GS>
__global__ __launch_bounds__(THREADS, 1) void k_gemm_w4a4_grouped_e3m2(GemmArgs a)
{
    using C = GroupRing6<GS>;
    static_assert(GS == 128 || GS == 256, "one or two k-blocks per group");
    extern __shared__ __align__(16) uint8_t lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;  // 64 x 64 wave tiles
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + BM - 1) / BM, TN = (N + GBN - 1) / GBN;
    const int T = TM * TN;
    const int G = gridDim.x, b = blockIdx.x;
    const int KT = K / 128;

    const bool xcd = (G % 8 == 0) && (T % 8 == 0) && G <= T;
    auto tile_pos = [&](int it) -> int {
        if (xcd) {
            const int per_x = T / 8, gx = G / 8;
            const int r = (b >> 3) + it * gx;
            return r < per_x ? (b & 7) * per_x + r : -1;
        }
        const int t = b + it * G;
        return t < T ? t : -1;
    };
    // tiles in groups of 4 m-tiles: the 32 concurrent 256 x 128 tiles of an
    // XCD then cover 4 X and 8 W panels (2048 rows) instead of 8 X and 4 W
    // (2560 rows) with groups of 8, 20% fewer bytes through its L2
    // (Llama-2-70B down shape, K = 28672: 4.45 -> 4.27 ms at G = 128)
    constexpr int GM4 = 4;
    auto tile_mn = [&](int t, int &m0, int &n0) {
        const int gsize = GM4 * TN;
        const int g = t / gsize;
        const int first = g * GM4;
        const int gm = min(TM - first, GM4);
        const int r = t - g * gsize;
        m0 = (first + r % gm) * BM;
        n0 = (r / gm) * GBN;
    };

    // Operand DMAs in the SGPR-base form: a per-lane 32-bit offset inside
    // the tile's run of heads (row lane / 4, 16-byte unit lane % 4) or tails
    // (row lane / 2, half lane % 2), rows past the matrix edge clamped, fixed
    // per tile; and wave-uniform bases, advanced by one k-block per step.
    const bool wtail = wave < 4;  // DMA 4 moves W tails (else scales)
    uint32_t vo[5];
    auto set_voff = [&](int m0, int n0) {
        const int xl = M - 1 - m0, wl = N - 1 - n0;
        vo[0] = (uint32_t)(min(16 * wave + (lane >> 2), xl) * 64 + (lane & 3) * 16);
        vo[1] = (uint32_t)(min(128 + 16 * wave + (lane >> 2), xl) * 64 + (lane & 3) * 16);
        vo[2] = (uint32_t)(min(16 * wave + (lane >> 2), wl) * 64 + (lane & 3) * 16);
        vo[3] = (uint32_t)(min(32 * wave + (lane >> 1), xl) * 32 + (lane & 1) * 16);
        vo[4] = (uint32_t)(min(32 * (wave & 3) + (lane >> 1), wl) * 32 + (lane & 1) * 16);
    };
    const int64_t xblk = (int64_t)M * 96, wblk = (int64_t)N * 96;
    const uint8_t *bxh, *bwh, *bxt, *bwt;  // bases of the next DMA step
    auto set_base = [&](int m0, int n0, int sk) {
        bxh = a.xq + sk * xblk + (int64_t)m0 * 64;
        bwh = a.wq + sk * wblk + (int64_t)n0 * 64;
        bxt = a.xq + sk * xblk + (int64_t)M * 64 + (int64_t)m0 * 32;
        bwt = a.wq + sk * wblk + (int64_t)N * 64 + (int64_t)n0 * 32;
    };
    const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_void *)lds;
    // scale load of waves 4-7 for k-step sk of the tile at (m0, n0): 2 fp16
    // per lane, the element index clamped to an even one inside the vector
    const int part = wave - 4;
    auto scale_src = [&](int m0, int n0, int sk) -> const uint16_t * {
        const int64_t g = sk / C::GST;
        if (part < 2)
            return a.sx + g * M + min(m0 + 128 * part + 2 * lane, M - 2);
        return a.sw + g * N + min(n0 + 2 * lane, N - 2);
    };
    auto issue = [&](int sm0, int sn0, int sk, int stage) {
        const uint32_t sb = lds_base + stage * C::STAGE;
        dma16s(vo[0], bxh, sb + wave * 1024);
        dma16s(vo[1], bxh, sb + (wave + 8) * 1024);
        dma16s(vo[2], bwh, sb + (wave + 16) * 1024);
        dma16s(vo[3], bxt, sb + C::HEADS + wave * 1024);
        if (wtail)
            dma16s(vo[4], bwt, sb + C::HEADS + (wave + 8) * 1024);
        else
            dma4(scale_src(sm0, sn0, sk), sb + C::SCL + part * 256);
    };
    auto advance = [&]() {
        bxh += xblk;
        bwh += wblk;
        bxt += xblk;
        bwt += wblk;
    };

    // LDS reads: X slice j (MFMA B operand) = stage rows wm 64 + 16 j + orow,
    // W slice i (A operand) = stage rows BM + wn 64 + 16 i + orow; lane group
    // q takes unit q of the 128-k block: its head at slot q ^ ((r >> 1) & 3),
    // its tail at slot q ^ ((r >> 2) & 3) (slices start at multiples of 16)
    const int orow = lane & 15, q = lane >> 4;
    const int hsl = (q ^ ((orow >> 1) & 3)) << 4, tsl = 8 * (q ^ ((orow >> 2) & 3));
    const int xh = (wm * 64 + orow) * 64 + hsl, xt = C::HEADS + (wm * 64 + orow) * 32 + tsl;
    const int wh = (BM + wn * 64 + orow) * 64 + hsl;
    const int wt = C::HEADS + (BM + wn * 64 + orow) * 32 + tsl;
    auto rd = [&](const uint8_t *sb, int h, int t) -> Op6 {
        Op6 o;
        o.h = *reinterpret_cast<const uint4 *>(sb + h);
        const uint64_t v = *(const volatile lds_u64 *)(lds_void *)(sb + t);
        o.t = make_uint2((uint32_t)v, (uint32_t)(v >> 32));
        return o;
    };

    int t = tile_pos(0);
    if (t < 0)
        return;
    int m0, n0;
    tile_mn(t, m0, n0);
    set_voff(m0, n0);
    // global step g of this block lives in stage g % RS.  A step's operands
    // are read from LDS during the step before it, so before step g starts
    // the loads of step g + 1 must have landed for every wave: only the
    // latest step's D loads stay in flight across a barrier.
#pragma unroll
    for (int s = 0; s < C::RS - 1; ++s) {
        set_base(m0, n0, min(s, KT - 1));
        issue(m0, n0, min(s, KT - 1), s);
    }
    set_base(m0, n0, C::RS - 1);
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((C::RS - 3) * C::D, 15));
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
    Op6 X[4], W[4];
    auto read_ops = [&](const uint8_t *sb) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            X[j] = rd(sb, xh + j * 16 * 64, xt + j * 16 * 32);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            W[i] = rd(sb, wh + i * 16 * 64, wt + i * 16 * 32);
    };
    read_ops(lds);

    int g = 0;
    for (int it = 0; t >= 0; ++it) {
        const int tn_ = tile_pos(it + 1);
        int m1 = 0, n1 = 0;
        if (tn_ >= 0)
            tile_mn(tn_, m1, n1);

        float yacc[4][4][4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    yacc[j][i][r] = 0.0f;
        v4f tt[4][4];

        // one k-step; FIRST: the group's first (temporaries start at 0),
        // LAST: its last (dequantize into yacc)
        auto step = [&](int kt, auto FIRST, auto LAST) {
            // DMA of global step g + RS - 1 into the stage of step g - 1
            // (read during step g - 2): this tile's step kt + RS - 1, else
            // the next tile's, else (no next tile) a harmless re-fetch
            {
                const bool here = kt + C::RS - 1 < KT;
                const int stage = (g + C::RS - 1) % C::RS;
                if (here || tn_ >= 0) {
                    const int sk = here ? kt + C::RS - 1 : kt + C::RS - 1 - KT;
                    if (kt + C::RS - 1 == KT) {
                        set_voff(m1, n1);
                        set_base(m1, n1, 0);
                    }
                    issue(here ? m0 : m1, here ? n0 : n1, sk, stage);
                    advance();
                } else {
                    set_base(m0, n0, KT - 1);
                    issue(m0, n0, KT - 1, stage);
                }
            }
            const uint8_t *sb = lds + (g % C::RS) * C::STAGE;
            // this step's scales (read first: LDS reads complete in order),
            // sx of the lane's row per X slice, sw of its four columns per W
            // slice
            // (kept as fp16: the multiplies take them as mixed-precision
            // operands, so no conversions)
            _Float16 sxv[4], swv[4][4];
            if constexpr (decltype(LAST)::value) {
                const _Float16 *lsc = reinterpret_cast<const _Float16 *>(sb + C::SCL);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    sxv[j] = lsc[wm * 64 + j * 16 + orow];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint2 w2 =
                        *reinterpret_cast<const uint2 *>(lsc + 256 + wn * 64 + i * 16 + q * 4);
                    swv[i][0] = __builtin_bit_cast(_Float16, (uint16_t)w2.x);
                    swv[i][1] = __builtin_bit_cast(_Float16, (uint16_t)(w2.x >> 16));
                    swv[i][2] = __builtin_bit_cast(_Float16, (uint16_t)w2.y);
                    swv[i][3] = __builtin_bit_cast(_Float16, (uint16_t)(w2.y >> 16));
                }
            }
            static_for<4>([&](auto JI) {
                constexpr int j = decltype(JI)::value;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    tt[j][i] = mfma6(W[i], X[j], decltype(FIRST)::value ? v4f{0.0f, 0.0f, 0.0f, 0.0f}
                                                                        : tt[j][i]);
            });
            __builtin_amdgcn_sched_barrier(0);
            // the next step's operands into the same registers (the MFMAs
            // above have taken theirs); their latency runs under the dequant
            read_ops(lds + ((g + 1) % C::RS) * C::STAGE);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (decltype(LAST)::value) {
                // per X slice, in three batches of 16 independent operations
                // (multiply by sx, multiply by sw, add), so that consecutive
                // VALU instructions of a wave do not wait on each other; each
                // output still takes RN(RN(acc sx) sw), then one add
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    float u[4][4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            u[i][r] = mul_h(tt[j][i][r], sxv[j]);
                    __asm__ volatile("" : "+v"(u[0][0]), "+v"(u[0][1]), "+v"(u[0][2]), "+v"(u[0][3]),
                                     "+v"(u[1][0]), "+v"(u[1][1]), "+v"(u[1][2]), "+v"(u[1][3]),
                                     "+v"(u[2][0]), "+v"(u[2][1]), "+v"(u[2][2]), "+v"(u[2][3]),
                                     "+v"(u[3][0]), "+v"(u[3][1]), "+v"(u[3][2]), "+v"(u[3][3]));
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            u[i][r] = mul_h(u[i][r], swv[i][r]);
                    __asm__ volatile("" : "+v"(u[0][0]), "+v"(u[0][1]), "+v"(u[0][2]), "+v"(u[0][3]),
                                     "+v"(u[1][0]), "+v"(u[1][1]), "+v"(u[1][2]), "+v"(u[1][3]),
                                     "+v"(u[2][0]), "+v"(u[2][1]), "+v"(u[2][2]), "+v"(u[2][3]),
                                     "+v"(u[3][0]), "+v"(u[3][1]), "+v"(u[3][2]), "+v"(u[3][3]));
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            yacc[j][i][r] = yacc[j][i][r] + u[i][r];
                            __asm__ volatile("" : "+v"(yacc[j][i][r]));
                        }
                }
            }
            // step g + 2 landed for this wave's loads (only step g + RS - 1
            // may stay in flight; loads complete in order), every LDS read
            // done; then for every wave
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm((C::RS - 3) * C::D, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
            ++g;
        };
        for (int kt = 0; kt < KT; kt += C::GST) {
            if constexpr (C::GST == 1) {
                step(kt, std::true_type{}, std::true_type{});
            } else {
                step(kt, std::true_type{}, std::false_type{});
                step(kt + 1, std::false_type{}, std::true_type{});
            }
        }

        // epilogue: lane holds n = nb + r (r < 4) of m = mb + orow per slice
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + j * 16 + orow;
            if (m >= M)
                continue;
            uint16_t *yrow = a.y + (int64_t)m * N;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int nb = n0 + wn * 64 + i * 16 + q * 4;
                if (nb >= N)
                    continue;  // N is a multiple of 8: a quad is all in or all out
                const h2 lo = __builtin_convertvector((f2){yacc[j][i][0], yacc[j][i][1]}, h2);
                const h2 hi = __builtin_convertvector((f2){yacc[j][i][2], yacc[j][i][3]}, h2);
                uint2 pk;
                pk.x = __builtin_bit_cast(uint32_t, lo);
                pk.y = __builtin_bit_cast(uint32_t, hi);
                *reinterpret_cast<uint2 *>(yrow + nb) = pk;
            }
        }

        t = tn_;
        m0 = m1;
        n0 = n1;
    }
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));  // no DMA may outlive the block's LDS
}
}  // namespace

namespace {
template <int GS>
hipError_t gemm_grouped_as(const GemmArgs &a, hipStream_t s)
{
    if (a.K % GroupTile<GS>::KS)
        return hipErrorInvalidValue;
    const int TM = (a.M + BM - 1) / BM, TN = (a.N + GBN - 1) / GBN;
    const int tiles = TM * TN;
    if (a.M % 8 == 0 && a.N % 8 == 0) {
        // persistent ring kernel: one block per CU, or one per tile when
        // there are fewer tiles or fewer k-steps than ring stages
        using C = GroupRing<GS>;
        hipError_t e = hipFuncSetAttribute((const void *)k_gemm_w4a4_grouped_ring<GS>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
        if (e != hipSuccess)
            return e;
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        int grid = (tiles < cus || a.K / C::KS < C::RS) ? tiles : cus;
        if (grid >= 8 && tiles % 8 == 0)
            grid -= grid % 8;
        hipLaunchKernelGGL(k_gemm_w4a4_grouped_ring<GS>, dim3((unsigned)grid), dim3(THREADS),
                           C::LDS, s, a);
        return hipGetLastError();
    }
    using T = GroupTile<GS>;
    hipError_t e = hipFuncSetAttribute((const void *)k_gemm_w4a4_grouped<GS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_gemm_w4a4_grouped<GS>, dim3((unsigned)tiles), dim3(THREADS), T::LDS, s,
                       a);
    return hipGetLastError();
}

template <int GS>
hipError_t gemm_grouped_e3m2_as(const GemmArgs &a, hipStream_t s)
{
    using C = GroupRing6<GS>;
    if (a.K % GS || a.M % 8 || a.N % 8)
        return hipErrorInvalidValue;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + GBN - 1) / GBN);
    hipError_t e = hipFuncSetAttribute((const void *)k_gemm_w4a4_grouped_e3m2<GS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess)
        return e;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    // persistent: one block per CU, or one per tile when there are fewer
    // tiles or fewer k-steps than ring stages
    int grid = (tiles < cus || a.K / 128 < C::RS) ? tiles : cus;
    if (grid >= 8 && tiles % 8 == 0)
        grid -= grid % 8;
    hipLaunchKernelGGL(k_gemm_w4a4_grouped_e3m2<GS>, dim3((unsigned)grid), dim3(THREADS), C::LDS,
                       s, a);
    return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm_grouped(const GemmArgs &a, int group, hipStream_t s)
{
    if (a.M == 0 || a.N == 0)
        return hipSuccess;
    switch (group) {
    case 64: return gemm_grouped_as<64>(a, s);
    case 128: return gemm_grouped_as<128>(a, s);
    case 256: return gemm_grouped_as<256>(a, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemm_grouped_e3m2(const GemmArgs &a, int group, hipStream_t s)
{
    if (a.M == 0 || a.N == 0)
        return hipSuccess;
    switch (group) {
    case 128: return gemm_grouped_e3m2_as<128>(a, s);
    case 256: return gemm_grouped_e3m2_as<256>(a, s);
    }
    return hipErrorInvalidValue;
}
}  // namespace quarot
