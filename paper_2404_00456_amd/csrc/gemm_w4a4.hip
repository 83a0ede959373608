// W4A4 integer GEMM with fused dequant epilogue (§4 Stage 2b, App. A.10),
// for gfx950.
//
//   acc[m][n] = sum_k qx[m][k] qw[n][k]                       (int32, exact)
//   y[m][n]   = RN16(RN(RN(float(acc) * sx[m]) * sw[n]))
//
// gfx950 has no int4 matrix instruction, so the packed codes are widened to
// int8 and fed to v_mfma_i32_16x16x64_i8.  Widening puts each nibble in the
// high half of a byte (value 16 q, two's complement intact): the low nibbles
// of a packed dword d become (d << 4) & 0xF0F0F0F0 and the high nibbles
// d & 0xF0F0F0F0.  The products then carry a factor 256, removed exactly by
// an arithmetic shift (|256 acc| <= 256 * 64 * 65536 < 2^31).  Both operands
// get the same permutation of k within each 64-wide slice, which leaves the
// dot products unchanged.
//
// Tiling: a block computes 256 (m) x 256 (n) with eight waves of 128 x 64
// (two waves per SIMD, 128 accumulator registers each).
// Each k-step stages 128 k (64 packed bytes per row) of both operands in
// LDS, double buffered; rows are padded to 80 bytes so the 8-byte operand
// reads of 16 consecutive rows hit distinct banks.  The W tile is the MFMA
// A operand and the X tile the B operand, so each lane ends up holding four
// consecutive n of one m: the epilogue stores 8 bytes of y per lane.
// Blocks are numbered XCD by XCD (the dispatcher deals blocks to the eight
// XCDs round-robin) and, within an XCD, in groups of 8 m-tiles, so blocks
// that share an L2 also share operand panels.
#include "common.hpp"

namespace quarot {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int BM = 256;   // X rows per block
constexpr int BN = 256;   // W rows per block
constexpr int BKB = 64;   // packed bytes per row per k-step
constexpr int LDSR = 80;  // LDS row pitch (bytes)
constexpr int GM = 8;     // m-tiles per group in the tile order
constexpr int STAGE = (BM + BN) * LDSR;
constexpr int LDS_BYTES = 2 * STAGE;

__device__ __forceinline__ v4i widen(uint2 d)
{
    v4i r;
    r[0] = (int)((d.x << 4) & 0xF0F0F0F0u);
    r[1] = (int)(d.x & 0xF0F0F0F0u);
    r[2] = (int)((d.y << 4) & 0xF0F0F0F0u);
    r[3] = (int)(d.y & 0xF0F0F0F0u);
    return r;
}

__device__ __forceinline__ void tile_of(int bid, int nblk, int TM, int TN, int &tm, int &tn)
{
    int t = bid;
    if ((nblk & 7) == 0)
        t = (bid & 7) * (nblk >> 3) + (bid >> 3);
    const int gsize = GM * TN;
    const int g = t / gsize;
    const int first = g * GM;
    const int gm = min(TM - first, GM);
    const int r = t - g * gsize;
    tm = first + r % gm;
    tn = r / gm;
}

constexpr int THREADS = 512;
constexpr int WN = 64;   // n per wave
constexpr int NI = WN / 16;  // n slices per wave (MFMA A operands)

__global__ __launch_bounds__(THREADS, 1) void k_gemm_w4a4(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + BM - 1) / BM, TN = (N + BN - 1) / BN;
    int tm, tn;
    tile_of(blockIdx.x, gridDim.x, TM, TN, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int64_t ldk = K / 2;  // packed row pitch in global memory
    const int KT = (K + 127) / 128;
    const bool tail = (K & 127) != 0;  // last k-step holds 64 k only

    // global -> LDS mapping: 16-byte chunk id = tid + 512 i, 4 chunks per row
    constexpr int NL = (BM * BKB / 16) / THREADS;  // chunks per thread per operand
    const uint8_t *gx[NL];
    const uint8_t *gw[NL];
    int lrow[NL], lcol[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
        const int id = tid + THREADS * i;
        lrow[i] = id >> 2;
        lcol[i] = id & 3;
        const int mr = min(m0 + lrow[i], M - 1);
        const int nr = min(n0 + lrow[i], N - 1);
        gx[i] = a.xq + (int64_t)mr * ldk + lcol[i] * 16;
        gw[i] = a.wq + (int64_t)nr * ldk + lcol[i] * 16;
    }

    uint4 px[NL], pw[NL];
    auto gload = [&](int kt) {
        const bool half = tail && kt == KT - 1;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            if (half && lcol[i] >= 2) {
                px[i] = make_uint4(0, 0, 0, 0);
                pw[i] = make_uint4(0, 0, 0, 0);
            } else {
                px[i] = *reinterpret_cast<const uint4 *>(gx[i] + (int64_t)kt * BKB);
                pw[i] = *reinterpret_cast<const uint4 *>(gw[i] + (int64_t)kt * BKB);
            }
        }
    };
    auto lstore = [&](int stage) {
        uint8_t *base = lds + stage * STAGE;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
            *reinterpret_cast<uint4 *>(base + lrow[i] * LDSR + lcol[i] * 16) = px[i];
            *reinterpret_cast<uint4 *>(base + (BM + lrow[i]) * LDSR + lcol[i] * 16) = pw[i];
        }
    };

    v4i acc[NI][8];
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = v4i{0, 0, 0, 0};

    gload(0);
    lstore(0);
    __syncthreads();

    const int orow = lane & 15;           // operand row within a 16-row slice
    const int obyte = (lane >> 4) * 8;    // operand bytes within a 32-byte k slice
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT)
            gload(kt + 1);
        const uint8_t *sb = lds + cur * STAGE;
        // a 64-wide k tail was zero-filled in LDS: both halves always run
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            v4i bq[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint8_t *p = sb + (wm * 128 + j * 16 + orow) * LDSR + kk * 32 + obyte;
                bq[j] = widen(*reinterpret_cast<const uint2 *>(p));
            }
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const uint8_t *p =
                    sb + (BM + wn * WN + i * 16 + orow) * LDSR + kk * 32 + obyte;
                const v4i aq = widen(*reinterpret_cast<const uint2 *>(p));
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aq, bq[j], acc[i][j], 0, 0, 0);
            }
        }
        if (kt + 1 < KT)
            lstore(cur ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds n = nb + 4*(lane>>4) + r (r = 0..3) of m = mb + (lane&15)
    float sxf[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int m = m0 + wm * 128 + j * 16 + orow;
        sxf[j] = h2f(a.sx[min(m, M - 1)]);
    }
    const bool vec = (N & 3) == 0;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        const int nb = n0 + wn * WN + i * 16 + (lane >> 4) * 4;
        float swf[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
            swf[r] = h2f(a.sw[min(nb + r, N - 1)]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int m = m0 + wm * 128 + j * 16 + orow;
            if (m >= M)
                continue;
            int iv[4];
            uint16_t hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                iv[r] = acc[i][j][r] >> 8;
                const float t = (float)iv[r] * sxf[j];
                hv[r] = f2h(t * swf[r]);
            }
            uint16_t *yrow = a.y + (int64_t)m * N;
            int32_t *arow = a.acc ? a.acc + (int64_t)m * N : nullptr;
            if (vec && nb + 3 < N) {
                uint2 pk;
                pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                *reinterpret_cast<uint2 *>(yrow + nb) = pk;
                if (arow)
                    *reinterpret_cast<int4 *>(arow + nb) = make_int4(iv[0], iv[1], iv[2], iv[3]);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (nb + r < N) {
                        yrow[nb + r] = hv[r];
                        if (arow)
                            arow[nb + r] = iv[r];
                    }
            }
        }
    }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s)
{
    if (a.M == 0 || a.N == 0)
        return hipSuccess;
    // more than 64 KB of dynamic LDS: raise the kernel's limit (per call, so
    // that every device the caller uses gets it; the call is host-side only)
    hipError_t e = hipFuncSetAttribute((const void *)k_gemm_w4a4,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
    if (e != hipSuccess)
        return e;
    const int TM = (a.M + BM - 1) / BM, TN = (a.N + BN - 1) / BN;
    hipLaunchKernelGGL(k_gemm_w4a4, dim3((unsigned)(TM * TN)), dim3(THREADS), LDS_BYTES, s, a);
    return hipGetLastError();
}

}  // namespace quarot
