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
#include "gemm_common.hpp"
#include "gemm_plan.hpp"

namespace quarot {
namespace {

using namespace gemm;

__global__ __launch_bounds__(THREADS, 1) void k_gemm_w4a4_k64(GemmArgs a)
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


// ------------------------------------------------------------------------
// Main kernel (K a multiple of 128).  Same block tile, waves and epilogue as
// the fallback above; the operand path differs:
//
//  * HBM -> LDS with global_load_lds_dwordx4 (no VGPR staging) into a ring
//    of S stages, three k-steps ahead of the MFMAs, one barrier per k-step.
//  * k assignment: within a k-step (128 k = 64 packed bytes per row), lane
//    group g = lane/16 of an operand owns the 16-byte unit g of its row and
//    uses its first 8 bytes in MFMA substep 0 and the last 8 in substep 1.
//    Every byte of the row is used once, by the same lane slot in A and B,
//    so the dot products are unchanged, and each operand is a single
//    ds_read_b128 per k-step.
//  * LDS rows are unpadded (the DMA writes a wave's lanes contiguously:
//    1 KB = 16 rows x 64 B); unit c of row r sits at unit c ^ ((r >> 1) & 3),
//    which makes the 16-byte reads of 8 consecutive rows hit 8 distinct bank
//    groups.
constexpr int S = 3;  // LDS ring stages
// Block tiles: TBM (m) x BN (n), TBM = 256 (eight waves) or 128 (four
// waves, for grids too small to give every compute unit a 256 x 256 tile);
// every wave computes 128 (m) x 64 (n).
template <int TBM>
struct Tile {
    static constexpr int NW = TBM / 128 * (BN / WN);  // waves
    static constexpr int THREADS = 64 * NW;
    static constexpr int HEADS = (TBM + BN) * 64;     // e3m2 stage: offset of the tails
    // Scales of a tile (TBM sx then BN sw, fp16) live in LDS after the ring,
    // double buffered by tile parity.
    static constexpr int SCALE_BYTES = 2 * (TBM + BN) * 2;
};

// Per code format: bytes per row per k-step, stage and ring sizes, DMAs per
// wave per k-step.  4- and 8-bit codes: 64 bytes per row (32 KB stages for
// 256 x 256 tiles).  e3m2 codes (BITS = 6): 96 bytes per row; a stage holds
// the 64-byte heads of all TBM + BN rows (X then W, laid out as the 4-bit
// stages), then their 32-byte tails (X then W).  DMA i < HPW of a wave moves
// a 1 KB chunk of heads (16 rows), the others a chunk of tails (32 rows).
template <int BITS, int TBM = 256>
struct Ring {
    static constexpr int KB = BITS == 6 ? 96 : 64;
    static constexpr int STAGE = (TBM + BN) * KB;
    static constexpr int BYTES = S * STAGE;
    static constexpr int HPW = (TBM + BN) * 64 / 1024 / Tile<TBM>::NW;
    static constexpr int DPW = STAGE / 1024 / Tile<TBM>::NW;
    static constexpr int LDS = BYTES + Tile<TBM>::SCALE_BYTES;
};

template <int BITS>
struct AccOf {
    typedef v4i type;
};
template <>
struct AccOf<6> {
    typedef v4f type;
};

// acc as int32 (4-bit codes: the accumulators hold 256 acc)
template <int BITS, typename T>
__device__ __forceinline__ int acc_int(T v)
{
    if constexpr (BITS == 4)
        return v >> 8;
    else if constexpr (BITS == 6)
        return (int)v;
    else
        return v;
}


// Persistent: each block walks a range of tiles.  Block b sits on XCD b % 8
// (the dispatcher deals blocks round-robin), so the 8 XCDs own contiguous
// eighths of the tile order and the blocks of one XCD take consecutive
// tiles, as the one-tile-per-block kernel above does.  The ring keeps
// running across tiles: the last S k-steps of a tile issue the DMAs of the
// next tile's first S, which land during the epilogue.  That needs at least
// S k-steps per tile; the launcher gives every block a single tile
// otherwise.
//
// BITS = 8 (codes of 6 or 8 bits, one byte each): the same ring, tiles and
// epilogue, but a k-step is 64 k (64 bytes per row), each 16-byte LDS read
// is one MFMA operand as it is (no widening), and the accumulators hold acc
// itself (no factor 256).  The 32 MFMAs of a k-step split into two halves
// around the barrier, as the two substeps of the 4-bit path do.
//
// BITS = 6 (int4 codes stored as e3m2, see k_pack_e3m2): a k-step is 128 k
// (96 bytes per row), one v_mfma_f32_16x16x128_f8f6f4 per 16x16 slice pair
// (half the MFMA count of the 4-bit path, no widening), binary32
// accumulators holding acc exactly.  Lane group g of an operand takes unit
// g (its 16-byte head and 8-byte tail), the same k in A and B.
template <int BITS, int TBM = 256>
__device__ __forceinline__ void gemm_main(const GemmArgs &a, uint8_t *lds)
{
    static_assert(BITS == 4 || BITS == 6 || BITS == 8, "int4, e3m2 or int8 codes");
    static_assert(TBM == 256 || TBM == 128, "block tile 256 or 128 rows");
    typedef Ring<BITS, TBM> R;
    typedef Tile<TBM> TL;
    constexpr int KB = R::KB;
    constexpr int DPW = R::DPW;
    constexpr int HPW = R::HPW;
    constexpr int NW = TL::NW;
    constexpr int HEADS = TL::HEADS;
    constexpr int SCALE_BYTES = TL::SCALE_BYTES;
    constexpr int RING_STAGE = R::STAGE;
    constexpr int RING_BYTES = R::BYTES;
    typedef typename AccOf<BITS>::type Acc;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + TBM - 1) / TBM, TN = (N + BN - 1) / BN;
    const int T = TM * TN;
    const int G = gridDim.x, b = blockIdx.x;
    const int64_t ldk = BITS == 4 ? K / 2 : K;  // row pitch (4- and 8-bit codes)
    const int KT = BITS == 8 ? K / 64 : K / 128;

    // this block's tiles: logical positions b, b + G, ... within a
    // per-XCD ordering when the grid and the tile count allow it
    const bool xcd = (G % 8 == 0) && (T % 8 == 0) && G <= T;
    // With 256 blocks and tile counts that are multiples of 16 both ways the
    // chip works through 16 x 16-tile super-blocks, one per round: XCD x
    // takes the 4 (m) x 8 (n) sub-block (x % 4, x / 4) of it, its 32 blocks
    // one tile each, so an XCD's L2 serves 4 X and 8 W panels as in the
    // order below, while the whole chip touches 16 X and 16 W panels per
    // round instead of every X panel.  Rounds run along n within a row of
    // super-blocks, in alternating directions, so that the X panels of a
    // row and the W panels at its turns come back from the last-level cache.
    const bool sblk = G == 256 && TM % 16 == 0 && TN % 16 == 0;
    auto tile_pos = [&](int it) -> int {  // it-th tile of this block, or -1
        if (sblk)
            return it < T / 256 ? it * 256 + b : -1;
        if (xcd) {
            const int per_x = T / 8, gx = G / 8;
            const int r = (b >> 3) + it * gx;
            return r < per_x ? (b & 7) * per_x + r : -1;
        }
        const int t = b + it * G;
        return t < T ? t : -1;
    };
    auto tile_mn = [&](int t, int &m0, int &n0) {
        if (sblk) {
            const int r = t >> 8, x = t & 7, s = (t >> 3) & 31;
            const int nsb = TN / 16, mb = r / nsb, nr = r - mb * nsb;
            const int nb = (mb & 1) ? nsb - 1 - nr : nr;
            m0 = (mb * 16 + (x & 3) * 4 + (s & 3)) * TBM;
            n0 = (nb * 16 + (x >> 2) * 8 + (s >> 2)) * BN;
            return;
        }
        const int gsize = GM * TN;
        const int g = t / gsize;
        const int first = g * GM;
        const int gm = min(TM - first, GM);
        const int r = t - g * gsize;
        m0 = (first + r % gm) * TBM;
        n0 = (r / gm) * BN;
    };

    // DMA sources.  Head DMA i < HPW of wave w moves chunk c = w + NW i of
    // the stage's heads: rows 16 c .. 16 c + 15 of the TBM X rows followed by
    // the BN W rows (the first two of every wave are X chunks), row
    // 16 c + lane/4 at unit lane%4 of its LDS row, so that it fetches global
    // unit (lane%4) ^ swizzle(row).  e3m2 operands (tiled layout, see
    // k_pack_e3m2): heads are already swizzled in memory, so lane l fetches
    // unit l % 4 of its row; the remaining DMAs i = HPW + j move tail chunk
    // c = w + NW j: rows 32 c + lane/2, 16 bytes each (the first of every
    // wave is an X chunk).  Every instruction reads 1 KB of consecutive bytes
    // (rows past the matrix edge are clamped).
    const int rsub = lane >> 2;
    const int cunit = (lane & 3) ^ ((lane >> 3) & 3);
    static_assert(DPW == (BITS == 6 ? HPW + HPW / 2 : HPW), "heads (+ tails) per wave");
    static_assert(TBM / 16 == 2 * NW && TBM / 32 == NW, "X chunks come first in every wave");
    auto is_x = [&](int i) { return i < 2 || i == HPW; };  // compile-time after unrolling
    auto chunk_row = [&](int i) -> int {  // first row of DMA i's chunk in its operand
        const int c = wave + NW * (i < HPW ? i : i - HPW);
        const int r = i < HPW ? 16 * c : 32 * c;
        return is_x(i) ? r : r - TBM;
    };
    int dst[DPW];
#pragma unroll
    for (int i = 0; i < DPW; ++i)
        dst[i] = i < HPW ? (wave + NW * i) * 1024 : HEADS + (wave + NW * (i - HPW)) * 1024;
    // e3m2 DMAs in the SGPR-base form.  voff6: lane offset of DMA i inside
    // the tile's run of heads (or tails), rows past the matrix edge clamped;
    // base6: the run's wave-uniform start for k-step sk.
    //
    // 4- and 8-bit codes (row-major, pitch ldk) use the same form: lane
    // offset r * ldk + unit (rows clamped), base x + m0 * ldk + sk * 64.
    auto voff6 = [&](int i, int m0, int n0) -> uint32_t {
        const bool xop = is_x(i);
        const int lim = (xop ? M - m0 : N - n0) - 1;
        if (i < HPW) {
            const int r = chunk_row(i) + rsub;
            if constexpr (BITS != 6)
                return (uint32_t)(min(r, lim) * (int)ldk + cunit * 16);
            return (uint32_t)(min(r, lim) * 64 + (lane & 3) * 16);
        }
        const int r = chunk_row(i) + (lane >> 1);
        return (uint32_t)(min(r, lim) * 32 + (lane & 1) * 16);
    };
    auto base6 = [&](int i, int m0, int n0, int sk) -> const uint8_t * {
        const bool xop = is_x(i);
        const int64_t org = xop ? m0 : n0;
        if constexpr (BITS != 6)
            return (xop ? a.xq : a.wq) + org * ldk + (int64_t)sk * BKB;
        const int64_t rows = xop ? M : N;
        const uint8_t *blk = (xop ? a.xq : a.wq) + (int64_t)sk * (rows * 96);
        return i < HPW ? blk + org * 64 : blk + rows * 64 + org * 32;
    };
    const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_void *)lds;
    int dsts[DPW];  // LDS targets, wave-uniform (scalar registers)
#pragma unroll
    for (int i = 0; i < DPW; ++i)
        dsts[i] = __builtin_amdgcn_readfirstlane(dst[i]);
    uint32_t vo[DPW];
    auto issue6 = [&](int m0, int n0, int sk, int stage) {
        const uint32_t sbase = lds_base + stage * RING_STAGE;
#pragma unroll
        for (int i = 0; i < DPW; ++i)
            dma16s(vo[i], base6(i, m0, n0, sk), sbase + dsts[i]);
    };
    // running bases of the next DMA step (wave-uniform), advanced by one
    // k-block per step: scalar adds instead of per-step products
    const uint8_t *bcur[DPW];
    auto stride6 = [&](int i) -> int64_t {
        return BITS == 6 ? (int64_t)(is_x(i) ? M : N) * 96 : (int64_t)BKB;
    };

    const int orow = lane & 15;
    const int ounit = ((lane >> 4) ^ ((orow >> 1) & 3)) << 4;
    const int brow = (wm * 128 + orow) * BKB + ounit;        // X slice rows (B operand)
    const int arow = (TBM + wn * WN + orow) * BKB + ounit;   // W slice rows (A operand)
    // e3m2 tails: the 8 bytes of unit g of row r sit at slot g ^ ((r >> 2) & 3)
    // of the row's 32-byte tail (16-row slices start at multiples of 16)
    const int toff = 8 * ((lane >> 4) ^ ((orow >> 2) & 3));
    const int btail = HEADS + (wm * 128 + orow) * 32 + toff;
    const int atail = HEADS + TBM * 32 + (wn * WN + orow) * 32 + toff;

    // Tiles wholly inside the matrices (and no int32 output) take the fast
    // epilogue, with the scales staged in LDS: one 4-byte DMA per wave, of
    // one 256-byte part (TBM / 128 parts of sx, then two of sw; with eight
    // waves, waves w and w + 4 fetch the same part, with four the fourth
    // fetches the first part again), issued ahead of the tile's operand DMAs
    // so that the k-loop's waits cover it.  Scale loads in the epilogue
    // itself would wait for the next tile's operand DMAs in flight (vmcnt is
    // in order).
    constexpr int XPARTS = TBM / 128, PARTS = XPARTS + 2;
    auto fast_tile = [&](int m0_, int n0_) {
        return m0_ + TBM <= M && n0_ + BN <= N && (N & 3) == 0 && a.acc == nullptr;
    };
    auto scale_dma = [&](int m0_, int n0_, int buf) {
        const int part = wave % PARTS;
        const uint16_t *gs = (part < XPARTS ? a.sx + m0_ + 128 * part
                                            : a.sw + n0_ + 128 * (part - XPARTS));
        dma4(gs + 2 * lane,
             __builtin_amdgcn_readfirstlane(lds_base + RING_BYTES + buf * (SCALE_BYTES / 2) +
                                            part * 256));
    };

    int t = tile_pos(0);
    if (t < 0)
        return;
    int m0, n0;
    tile_mn(t, m0, n0);
#pragma unroll
    for (int i = 0; i < DPW; ++i)
        vo[i] = voff6(i, m0, n0);
    if (fast_tile(m0, n0))
        scale_dma(m0, n0, 0);
    // ring position: global step g of this block lives in stage g % S
    int g = 0;
#pragma unroll
    for (int i = 0; i < S; ++i)
        issue6(m0, n0, min(i, KT - 1), i);
#pragma unroll
    for (int i = 0; i < DPW; ++i)
        bcur[i] = base6(i, m0, n0, S);

    for (int it = 0; t >= 0; ++it) {
        const int tn_ = tile_pos(it + 1);
        int m1 = 0, n1 = 0;
        if (tn_ >= 0)
            tile_mn(tn_, m1, n1);

        // The 128-row e3m2 tile (four waves, one per SIMD, accumulators in
        // AGPRs) does not clear its accumulators: its first k-step's MFMAs
        // take a zero accumulator operand instead (the compiler peels that
        // step), and the compiler then keeps the accumulators in place
        // through the loop, where it otherwise moved 24 of them per k-step
        // (M = 2048, N = 4096, K = 11008: 72 -> 64 us).  The 256-row tile measured
        // the same or 1% slower that way and clears.
        constexpr bool PEEL = BITS == 6 && TBM == 128;
        Acc acc[NI][8];
        if constexpr (!PEEL) {
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] = Acc{0, 0, 0, 0};
        }

        auto read_step = [&](uint4 (&ops)[8 + NI], int stage) {
            const uint8_t *sb = lds + stage * RING_STAGE;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                ops[j] = *reinterpret_cast<const uint4 *>(sb + brow + j * 16 * BKB);
#pragma unroll
            for (int i = 0; i < NI; ++i)
                ops[8 + i] = *reinterpret_cast<const uint4 *>(sb + arow + i * 16 * BKB);
        };
        auto substep = [&](const uint4 (&ops)[8 + NI], int h) {
            if constexpr (BITS == 4) {
                v4i aq[NI];
#pragma unroll
                for (int i = 0; i < NI; ++i)
                    aq[i] = widen(h ? make_uint2(ops[8 + i].z, ops[8 + i].w)
                                    : make_uint2(ops[8 + i].x, ops[8 + i].y));
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const v4i bq = widen(h ? make_uint2(ops[j].z, ops[j].w)
                                           : make_uint2(ops[j].x, ops[j].y));
#pragma unroll
                    for (int i = 0; i < NI; ++i)
                        acc[i][j] =
                            __builtin_amdgcn_mfma_i32_16x16x64_i8(aq[i], bq, acc[i][j], 0, 0, 0);
                }
            } else if constexpr (BITS == 8) {
                // half h: the B slices j = 4h .. 4h+3 against every A slice
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int j = 4 * h + jj;
                    const v4i bq = __builtin_bit_cast(v4i, ops[j]);
#pragma unroll
                    for (int i = 0; i < NI; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                            __builtin_bit_cast(v4i, ops[8 + i]), bq, acc[i][j], 0, 0, 0);
                }
            }
        };

        // Step 0 of this tile (global step g) must have landed for every
        // wave.  For the first tile: wait for it (S - 1 steps of DMAs stay in
        // flight) and synchronize.  For later tiles it was already waited
        // for, by every wave, before the last barrier of the previous tile
        // (and a wait here would also wait for the epilogue's stores, which
        // count in vmcnt).
        if (it == 0) {
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm((S - 1) * DPW, 15));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
        }
        if constexpr (BITS == 6) {
            // (A 4-wave variant, one wave per SIMD with 128 x 128 wave tiles
            // and the accumulators in AGPRs, reads a third less from LDS per
            // MFMA but measured ~5% slower on the Llama-2-70B FFN shapes:
            // one wave per SIMD exposes the latencies the second one hides.)
            //
            // A k-step is four quarters of 8 MFMAs over the slice pairs
            // A[0..1] x B[0..3], A[0..1] x B[4..7], A[2..3] x B[0..3],
            // A[2..3] x B[4..7].  Every read lands in registers a quarter
            // has just freed, at least one quarter before its first use, so
            // the operands are not double buffered:
            //   quarter 1: read B[4..7] of this step
            //   quarter 2: read A[2..3] of this step
            //   barrier after quarter 2 (every read of this stage done)
            //   quarter 3: read A[0..1] of the next step
            //   quarter 4: read B[0..3] of the next step
            // sched_barrier(0) fences keep that order: left to itself the
            // scheduler sinks each read to just before its first MFMA.
            // Within a quarter, sched_group_barrier interleaves its reads
            // with its MFMAs (1-4% faster than issuing them as one batch).
            Op6 A[NI], B[8];
            // tails read as volatile: the compiler would pair two slices'
            // tails into one ds_read2st64_b64 and then copy each next to its
            // head (the MFMA takes the six dwords as one register tuple)
            auto rdA = [&](int i, int stage) {
                const uint8_t *sb = lds + stage * RING_STAGE;
                A[i].h = *reinterpret_cast<const uint4 *>(sb + arow + i * 16 * 64);
                const uint64_t t = *(const volatile lds_u64 *)(lds_void *)(sb + atail + i * 16 * 32);
                A[i].t = make_uint2((uint32_t)t, (uint32_t)(t >> 32));
            };
            auto rdB = [&](int j, int stage) {
                const uint8_t *sb = lds + stage * RING_STAGE;
                B[j].h = *reinterpret_cast<const uint4 *>(sb + brow + j * 16 * 64);
                const uint64_t t = *(const volatile lds_u64 *)(lds_void *)(sb + btail + j * 16 * 32);
                B[j].t = make_uint2((uint32_t)t, (uint32_t)(t >> 32));
            };
            auto quarter = [&](int i0, int j0, bool first) {
#pragma unroll
                for (int i = i0; i < i0 + 2; ++i)
#pragma unroll
                    for (int j = j0; j < j0 + 4; ++j)
                        acc[i][j] = mfma6(A[i], B[j],
                                          PEEL && first ? v4f{0.0f, 0.0f, 0.0f, 0.0f} : acc[i][j]);
            };
            rdA(0, g % S);
            rdA(1, g % S);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                rdB(j, g % S);
            for (int kt = 0; kt < KT; ++kt, ++g) {
                const int cs = g % S, nx = (g + 1) % S;
#pragma unroll
                for (int j = 4; j < 8; ++j)
                    rdB(j, cs);
                quarter(0, 0, kt == 0);
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
                rdA(2, cs);
                rdA(3, cs);
                quarter(0, 4, kt == 0);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 3);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 3);
                __builtin_amdgcn_sched_barrier(0);
                __asm__ volatile("" ::: "memory");
                __builtin_amdgcn_s_waitcnt(waitcnt_imm((S - 2) * DPW, 0));
                __builtin_amdgcn_s_barrier();
                __asm__ volatile("" ::: "memory");
                {
                    // DMA of global step g+S: this tile's step kt+S, else the
                    // next tile's step kt+S-KT (its bases and lane offsets
                    // replace this tile's when the first of them is issued),
                    // else a harmless re-fetch (keeps the wait counts exact)
                    const uint32_t sbase = lds_base + (g % S) * RING_STAGE;
                    if (kt + S < KT || tn_ >= 0) {
                        if (kt + S == KT) {
#pragma unroll
                            for (int i = 0; i < DPW; ++i) {
                                vo[i] = voff6(i, m1, n1);
                                bcur[i] = base6(i, m1, n1, 0);
                            }
                        }
#pragma unroll
                        for (int i = 0; i < DPW; ++i) {
                            dma16s(vo[i], bcur[i], sbase + dsts[i]);
                            bcur[i] += stride6(i);
                        }
                    } else {
                        issue6(m0, n0, KT - 1, g % S);
                    }
                }
                rdA(0, nx);
                rdA(1, nx);
                quarter(2, 0, kt == 0);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    rdB(j, nx);
                quarter(2, 4, kt == 0);
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
        uint4 R[8 + NI], Rn[8 + NI];
        read_step(R, g % S);
        for (int kt = 0; kt < KT; ++kt, ++g) {
            substep(R, 0);
            // The s_waitcnt and s_barrier builtins do not order memory
            // accesses for the compiler; the empty asm statements do: every
            // LDS read of stage g is issued before the wait (and completes
            // by it), and no read of stage g+1 moves above the barrier.
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm((S - 2) * DPW, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
            // DMA of global step g+S: this tile's step kt+S, else the next
            // tile's step kt+S-KT (its bases and lane offsets replace this
            // tile's when the first of them is issued), else a harmless
            // re-fetch (keeps the wait counts exact)
            {
                const uint32_t sbase = lds_base + (g % S) * RING_STAGE;
                if (kt + S < KT || tn_ >= 0) {
                    if (kt + S == KT) {
#pragma unroll
                        for (int i = 0; i < DPW; ++i) {
                            vo[i] = voff6(i, m1, n1);
                            bcur[i] = base6(i, m1, n1, 0);
                        }
                    }
#pragma unroll
                    for (int i = 0; i < DPW; ++i) {
                        dma16s(vo[i], bcur[i], sbase + dsts[i]);
                        bcur[i] += stride6(i);
                    }
                } else {
                    issue6(m0, n0, KT - 1, g % S);
                }
            }
            read_step(Rn, (g + 1) % S);
            substep(R, 1);
#pragma unroll
            for (int o = 0; o < 8 + NI; ++o)
                R[o] = Rn[o];
        }
        }
        // the extra read after the last step touched stage g % S (the next
        // tile's step 0, landed) and is discarded

        // the next tile's scales: its buffer was last read by the epilogue
        // two tiles back, which every wave finished before this tile's
        // barriers
        if (tn_ >= 0 && fast_tile(m1, n1))
            scale_dma(m1, n1, (it + 1) & 1);

        if (fast_tile(m0, n0)) {
            // y = RN16(RN(RN(f32(acc) sx) sw)).  With 4-bit codes the
            // accumulators hold 256 acc and f32(256 acc) = 256 f32(acc), so
            // multiplying by sx / 256 (exact) gives the same RN(f32(acc) sx)
            // without the shift.
            const uint8_t *sc = lds + RING_BYTES + (it & 1) * (SCALE_BYTES / 2);
            const uint16_t *lsx = reinterpret_cast<const uint16_t *>(sc);
            const uint16_t *lsw = lsx + TBM;
            float sxs[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                sxs[j] = h2f(lsx[wm * 128 + j * 16 + orow]) * (BITS == 4 ? 0x1p-8f : 1.0f);
            float swf[NI][4];
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int nl = wn * WN + i * 16 + (lane >> 4) * 4;
                const uint2 swp = *reinterpret_cast<const uint2 *>(lsw + nl);
                swf[i][0] = h2f((uint16_t)swp.x);
                swf[i][1] = h2f((uint16_t)(swp.x >> 16));
                swf[i][2] = h2f((uint16_t)swp.y);
                swf[i][3] = h2f((uint16_t)(swp.y >> 16));
            }
            // row by row: the NI stores of one j cover 128 contiguous bytes
            // of each of 16 rows, back to back, so L2 lines fill at once
#pragma unroll
            for (int j = 0; j < 8; ++j) {
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    const int nl = wn * WN + i * 16 + (lane >> 4) * 4;
                    float u0 = ((float)acc[i][j][0] * sxs[j]) * swf[i][0];
                    float u1 = ((float)acc[i][j][1] * sxs[j]) * swf[i][1];
                    float u2 = ((float)acc[i][j][2] * sxs[j]) * swf[i][2];
                    float u3 = ((float)acc[i][j][3] * sxs[j]) * swf[i][3];
                    // pinned so the multiply is not fused into the conversion
                    __asm__ volatile("" : "+v"(u0), "+v"(u1), "+v"(u2), "+v"(u3));
                    const h2 lo = __builtin_convertvector((f2){u0, u1}, h2);
                    const h2 hi = __builtin_convertvector((f2){u2, u3}, h2);
                    uint2 pk;
                    pk.x = __builtin_bit_cast(uint32_t, lo);
                    pk.y = __builtin_bit_cast(uint32_t, hi);
                    const int m = m0 + wm * 128 + j * 16 + orow;
                    *reinterpret_cast<uint2 *>(a.y + (int64_t)m * N + n0 + nl) = pk;
                }
            }
        } else {
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
                    iv[r] = acc_int<BITS>(acc[i][j][r]);
                    const float tt = (float)iv[r] * sxf[j];
                    hv[r] = f2h(tt * swf[r]);
                }
                uint16_t *yrow = a.y + (int64_t)m * N;
                int32_t *arw = a.acc ? a.acc + (int64_t)m * N : nullptr;
                if (vec && nb + 3 < N) {
                    uint2 pk;
                    pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                    pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                    *reinterpret_cast<uint2 *>(yrow + nb) = pk;
                    if (arw)
                        *reinterpret_cast<int4 *>(arw + nb) = make_int4(iv[0], iv[1], iv[2], iv[3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (nb + r < N) {
                            yrow[nb + r] = hv[r];
                            if (arw)
                                arw[nb + r] = iv[r];
                        }
                }
            }
        }
        }

        t = tn_;
        m0 = m1;
        n0 = n1;
    }
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));  // no DMA may outlive the block's LDS
}

// ------------------------------------------------------------------------
// e3m2 operands, 128 (m) x 256 (n) block tiles, the k-steps of a tile split
// between two groups of four waves: group q takes the k-steps 2p + q
// (p = 0 .. KT/2 - 1, KT even), each of its waves 128 (m) x 64 (n) as in
// the kernel above, and the two partial sums meet in LDS at the end of the
// tile.  Both partials are integers of magnitude below 2^24 held exactly in
// binary32, so their sum is f32(acc) exactly.  Eight waves put two on each
// SIMD, which the 128-row tile of the kernel above (one wave per SIMD) does
// not: there the matrix cores idle while the single wave waits on its LDS
// reads and barriers.  For grids with too few 256 x 256 tiles to fill the
// chip.
//
// Ring: four 36 KB stages; k-step 2p + q in stage 2 (p % 2) + q, so each
// group double-buffers its own k-steps: the DMA of step 2p + q + 4 (issued by
// group q's waves after the barrier of pair p) must land by the barrier of
// pair p + 1, after which that step's first operands are read.  The ring does not run across tiles: at a tile's end it holds
// the 128 KB exchange of partial sums, then the next tile's first two pairs
// are issued before this tile's y stores.  Stage layout and DMA chunks are
// those of the 128-row tile above (four waves per group).
__device__ __forceinline__ void gemm_e3m2_ksplit(const GemmArgs &a, uint8_t *lds)
{
    constexpr int TBM = 128, NWG = 4;        // tile rows, waves per group
    constexpr int HEADS = (TBM + BN) * 64;   // offset of the tails in a stage
    constexpr int STAGE = (TBM + BN) * 96;   // 36 KB
    constexpr int HPW = HEADS / 1024 / NWG;  // 6 head DMAs per wave and step
    constexpr int DPW = STAGE / 1024 / NWG;  // 9 DMAs per wave and step
    static_assert(4 * STAGE >= 2 * NWG * 16 * 1024, "the exchange fits in the ring");
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = wave >> 2, wn = wave & 3;  // k group, n slice of the wave
    const int M = a.M, N = a.N, K = a.K;
    const int TM = (M + TBM - 1) / TBM, TN = (N + BN - 1) / BN;
    const int T = TM * TN;
    const int G = gridDim.x, b = blockIdx.x;
    const int P = K / 256;  // k-step pairs

    // tile order of the kernel above
    const bool xcd = (G % 8 == 0) && (T % 8 == 0) && G <= T;
    const bool sblk = G == 256 && TM % 16 == 0 && TN % 16 == 0;
    auto tile_pos = [&](int it) -> int {
        if (sblk)
            return it < T / 256 ? it * 256 + b : -1;
        if (xcd) {
            const int per_x = T / 8, gx = G / 8;
            const int r = (b >> 3) + it * gx;
            return r < per_x ? (b & 7) * per_x + r : -1;
        }
        const int t = b + it * G;
        return t < T ? t : -1;
    };
    auto tile_mn = [&](int t, int &m0, int &n0) {
        if (sblk) {
            const int r = t >> 8, x = t & 7, s = (t >> 3) & 31;
            const int nsb = TN / 16, mb = r / nsb, nr = r - mb * nsb;
            const int nb = (mb & 1) ? nsb - 1 - nr : nr;
            m0 = (mb * 16 + (x & 3) * 4 + (s & 3)) * TBM;
            n0 = (nb * 16 + (x >> 2) * 8 + (s >> 2)) * BN;
            return;
        }
        const int gsize = GM * TN;
        const int g = t / gsize;
        const int first = g * GM;
        const int gm = min(TM - first, GM);
        const int r = t - g * gsize;
        m0 = (first + r % gm) * TBM;
        n0 = (r / gm) * BN;
    };

    // DMAs of wave wn of group q for one k-step: head DMA i < HPW moves chunk
    // c = wn + 4 i of the stage's heads (rows 16 c .. 16 c + 15 of the 128 X
    // rows followed by the 256 W rows; i < 2 are X chunks), tail DMA
    // i = HPW + j chunk c = wn + 4 j of the tails (rows 32 c .. 32 c + 31;
    // j = 0 is the X chunk).  Lane offsets fixed per tile (rows past the
    // matrix edge clamped), wave-uniform bases advanced by two k-blocks per
    // pair.
    auto is_x = [&](int i) { return i < 2 || i == HPW; };
    auto chunk_row = [&](int i) -> int {
        const int c = wn + NWG * (i < HPW ? i : i - HPW);
        const int r = i < HPW ? 16 * c : 32 * c;
        return is_x(i) ? r : r - TBM;
    };
    // (el: the lane index, laundered by the caller so that nothing derived
    // from it is hoisted out of the tile loop and held through the k-loop)
    auto voff = [&](int i, int m0, int n0, int el) -> uint32_t {
        const int lim = (is_x(i) ? M - m0 : N - n0) - 1;
        if (i < HPW)
            return (uint32_t)(min(chunk_row(i) + (el >> 2), lim) * 64 + (el & 3) * 16);
        return (uint32_t)(min(chunk_row(i) + (el >> 1), lim) * 32 + (el & 1) * 16);
    };
    // four wave-uniform bases (X heads, W heads, X tails, W tails) of the
    // next k-step this group moves
    const int64_t xblk = (int64_t)M * 96, wblk = (int64_t)N * 96;
    const uint8_t *bxh, *bwh, *bxt, *bwt;
    auto set_base = [&](int m0, int n0, int sk) {
        bxh = a.xq + sk * xblk + (int64_t)m0 * 64;
        bwh = a.wq + sk * wblk + (int64_t)n0 * 64;
        bxt = a.xq + sk * xblk + (int64_t)M * 64 + (int64_t)m0 * 32;
        bwt = a.wq + sk * wblk + (int64_t)N * 64 + (int64_t)n0 * 32;
    };
    const uint32_t wdst = (uint32_t)(uintptr_t)(lds_void *)lds + wn * 1024;
    uint32_t vo[DPW];
    // one k-step of this wave's DMAs into the stage at LDS offset so
    auto issue = [&](int so) {
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const uint8_t *bs = i < HPW ? (is_x(i) ? bxh : bwh) : (is_x(i) ? bxt : bwt);
            const int d = i < HPW ? i * NWG * 1024 : HEADS + (i - HPW) * NWG * 1024;
            dma16s(vo[i], bs, wdst + so + d);
        }
    };
    auto advance2 = [&]() {
        bxh += 2 * xblk;
        bwh += 2 * wblk;
        bxt += 2 * xblk;
        bwt += 2 * wblk;
    };
    // the tile's first two pairs (k-steps q and 2 + q) into stages q, 2 + q
    auto start_tile = [&](int m0, int n0) {
        int el = lane;
        __asm__ volatile("" : "+v"(el));
#pragma unroll
        for (int i = 0; i < DPW; ++i)
            vo[i] = voff(i, m0, n0, el);
        set_base(m0, n0, q);
        issue(q * STAGE);
        advance2();
        issue((2 + q) * STAGE);
        advance2();
    };

    // LDS reads: X slice j (MFMA B operand) = stage row 16 j + orow, W slice
    // i (A operand) = stage row TBM + 64 wn + 16 i + orow; lane group lane/16
    // takes its unit of the 128-k block (head slot and tail slot swizzled as
    // k_pack_e3m2 lays them out)
    const int orow = lane & 15;
    const int ounit = ((lane >> 4) ^ ((orow >> 1) & 3)) << 4;
    const int toff = 8 * ((lane >> 4) ^ ((orow >> 2) & 3));
    const int brow = orow * 64 + ounit, arow = (TBM + wn * WN + orow) * 64 + ounit;
    const int btail = HEADS + orow * 32 + toff;
    const int atail = HEADS + TBM * 32 + (wn * WN + orow) * 32 + toff;
    Op6 A[NI], B[8];
    auto rdA = [&](int i, int stage) {
        const uint8_t *sb = lds + stage * STAGE;
        A[i].h = *reinterpret_cast<const uint4 *>(sb + arow + i * 16 * 64);
        const uint64_t t = *(const volatile lds_u64 *)(lds_void *)(sb + atail + i * 16 * 32);
        A[i].t = make_uint2((uint32_t)t, (uint32_t)(t >> 32));
    };
    auto rdB = [&](int j, int stage) {
        const uint8_t *sb = lds + stage * STAGE;
        B[j].h = *reinterpret_cast<const uint4 *>(sb + brow + j * 16 * 64);
        const uint64_t t = *(const volatile lds_u64 *)(lds_void *)(sb + btail + j * 16 * 32);
        B[j].t = make_uint2((uint32_t)t, (uint32_t)(t >> 32));
    };

    int t = tile_pos(0);
    if (t < 0)
        return;
    int m0, n0;
    tile_mn(t, m0, n0);
    start_tile(m0, n0);
    // vm operations this wave issued after the current tile's first pair:
    // its second pair, and the previous tile's y stores when they are known
    // to be 16 (else 0: wait for everything)
    int after = DPW;
    for (int it = 0; t >= 0; ++it) {
        const int tn_ = tile_pos(it + 1);
        int m1 = 0, n1 = 0;
        if (tn_ >= 0)
            tile_mn(tn_, m1, n1);

        v4f acc[NI][8];
#pragma unroll
        for (int i = 0; i < NI; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j)
                acc[i][j] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

        // pair 0 landed for every wave
        __asm__ volatile("" ::: "memory");
        if (after == DPW)
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(DPW, 15));
        else if (after == DPW + 16)
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(DPW + 16, 15));
        else
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));
        __builtin_amdgcn_s_barrier();
        __asm__ volatile("" ::: "memory");
        rdA(0, q);
        rdA(1, q);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            rdB(j, q);

        auto quarter = [&](int i0, int j0) {
#pragma unroll
            for (int i = i0; i < i0 + 2; ++i)
#pragma unroll
                for (int j = j0; j < j0 + 4; ++j)
                    acc[i][j] = mfma6(A[i], B[j], acc[i][j]);
        };
        // pair p: the quarters, reads and fences of the kernel above; LAST:
        // no next step to read
        auto pair = [&](int p, auto LAST) {
            const int cs = 2 * (p & 1) + q, nx = 2 * ((p + 1) & 1) + q;
#pragma unroll
            for (int j = 4; j < 8; ++j)
                rdB(j, cs);
            quarter(0, 0);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
            rdA(2, cs);
            rdA(3, cs);
            quarter(0, 4);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 3);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 3);
            __builtin_amdgcn_sched_barrier(0);
            // this wave's DMAs of pair p + 1 landed and its reads of stage
            // cs done; then for every wave
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
            if (p + 2 < P) {
                issue(cs * STAGE);
                advance2();
            }
            if constexpr (!decltype(LAST)::value) {
                rdA(0, nx);
                rdA(1, nx);
            }
            quarter(2, 0);
            if constexpr (!decltype(LAST)::value) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
            }
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (!decltype(LAST)::value) {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    rdB(j, nx);
            }
            quarter(2, 4);
            if constexpr (!decltype(LAST)::value) {
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        };
        for (int p = 0; p < P - 1; ++p)
            pair(p, std::false_type{});
        pair(P - 1, std::true_type{});

        // Every wave is past the last barrier: no ring reads or DMAs remain.
        // Group q finishes m rows 64 q .. 64 q + 63 of the tile (slices
        // j = 4 q .. 4 q + 3): the other group's partials of those rows come
        // through LDS, 1 KB per (wave, slice pair), both directions at once.
        // (QC: q as a compile-time constant, so that the accumulators are
        // indexed statically.)
        const bool fast = m0 + TBM <= M && n0 + BN <= N && (N & 3) == 0 && a.acc == nullptr;
        auto finish = [&](auto QC) {
            constexpr int Q = decltype(QC)::value, O = 1 - Q;
            // the lane's epilogue offsets are derived here, from a copy of
            // the lane index the compiler cannot see through: hoisted above
            // the k-loop they would be held (spilled) through it
            int el = lane;
            __asm__ volatile("" : "+v"(el));
            const int erow = el & 15, ecol = (el >> 4) * 4;
            float sxs[4];
            uint2 swp[NI];
            if (fast) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    sxs[jj] = h2f(a.sx[m0 + 64 * Q + 16 * jj + erow]);
#pragma unroll
                for (int i = 0; i < NI; ++i)
                    swp[i] = *reinterpret_cast<const uint2 *>(a.sw + n0 + wn * WN + i * 16 + ecol);
            }
            uint8_t *xw = lds + (O * NWG + wn) * 16 * 1024 + el * 16;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    *reinterpret_cast<v4f *>(xw + (i * 4 + jj) * 1024) = acc[i][4 * O + jj];
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");
            const uint8_t *xr = lds + (Q * NWG + wn) * 16 * 1024 + el * 16;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    acc[i][4 * Q + jj] += *reinterpret_cast<const v4f *>(xr + (i * 4 + jj) * 1024);
            __asm__ volatile("" ::: "memory");
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));
            __builtin_amdgcn_s_barrier();
            __asm__ volatile("" ::: "memory");

            if (fast) {
                // y = RN16(RN(RN(f32(acc) sx) sw)), packed before the next
                // tile's DMAs are issued (so the scale loads are waited for
                // alone) and stored after them
                uint2 pk[4][NI];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                    for (int i = 0; i < NI; ++i) {
                        const v4f v = acc[i][4 * Q + jj];
                        float u0 = (v[0] * sxs[jj]) * h2f((uint16_t)swp[i].x);
                        float u1 = (v[1] * sxs[jj]) * h2f((uint16_t)(swp[i].x >> 16));
                        float u2 = (v[2] * sxs[jj]) * h2f((uint16_t)swp[i].y);
                        float u3 = (v[3] * sxs[jj]) * h2f((uint16_t)(swp[i].y >> 16));
                        // pinned so the multiply is not fused into the conversion
                        __asm__ volatile("" : "+v"(u0), "+v"(u1), "+v"(u2), "+v"(u3));
                        const h2 lo = __builtin_convertvector((f2){u0, u1}, h2);
                        const h2 hi = __builtin_convertvector((f2){u2, u3}, h2);
                        pk[jj][i] = make_uint2(__builtin_bit_cast(uint32_t, lo),
                                               __builtin_bit_cast(uint32_t, hi));
                    }
                if (tn_ >= 0)
                    start_tile(m1, n1);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                    for (int i = 0; i < NI; ++i) {
                        const int m = m0 + 64 * Q + 16 * jj + erow;
                        const int nl = wn * WN + i * 16 + ecol;
                        *reinterpret_cast<uint2 *>(a.y + (int64_t)m * N + n0 + nl) = pk[jj][i];
                    }
                after = DPW + 16;
                return;
            }
            // edge tiles (and the int32 output): bounds per row and column
            const bool vec = (N & 3) == 0;
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int nb = n0 + wn * WN + i * 16 + ecol;
                float swf[4];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    swf[r] = h2f(a.sw[min(nb + r, N - 1)]);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int m = m0 + 64 * Q + 16 * jj + erow;
                    if (m >= M)
                        continue;
                    const float sxf = h2f(a.sx[m]);
                    int iv[4];
                    uint16_t hv[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        iv[r] = (int)acc[i][4 * Q + jj][r];
                        const float tt = (float)iv[r] * sxf;
                        hv[r] = f2h(tt * swf[r]);
                    }
                    uint16_t *yrow = a.y + (int64_t)m * N;
                    int32_t *arw = a.acc ? a.acc + (int64_t)m * N : nullptr;
                    if (vec && nb + 3 < N) {
                        uint2 pk;
                        pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                        pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                        *reinterpret_cast<uint2 *>(yrow + nb) = pk;
                        if (arw)
                            *reinterpret_cast<int4 *>(arw + nb) =
                                make_int4(iv[0], iv[1], iv[2], iv[3]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (nb + r < N) {
                                yrow[nb + r] = hv[r];
                                if (arw)
                                    arw[nb + r] = iv[r];
                            }
                    }
                }
            }
            if (tn_ >= 0)
                start_tile(m1, n1);
            after = 0;
        };
        if (q == 0)
            finish(std::integral_constant<int, 0>{});
        else
            finish(std::integral_constant<int, 1>{});
        t = tn_;
        m0 = m1;
        n0 = n1;
    }
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));  // no DMA may outlive the block's LDS
}

__global__ __launch_bounds__(Tile<256>::THREADS, 1) void k_gemm_w4a4(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<4>(a, lds);
}

__global__ __launch_bounds__(Tile<256>::THREADS, 1) void k_gemm_w8a8(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<8>(a, lds);
}

__global__ __launch_bounds__(Tile<256>::THREADS, 1) void k_gemm_w4a4_e3m2(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<6>(a, lds);
}

// 128 x 256 block tiles (four waves): for grids with too few 256 x 256
// tiles to keep every compute unit busy.
__global__ __launch_bounds__(Tile<128>::THREADS, 1) void k_gemm_w4a4_m128(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<4, 128>(a, lds);
}

__global__ __launch_bounds__(Tile<128>::THREADS, 1) void k_gemm_w8a8_m128(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<8, 128>(a, lds);
}

__global__ __launch_bounds__(Tile<128>::THREADS, 1) void k_gemm_w4a4_e3m2_m128(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_main<6, 128>(a, lds);
}

// 128 x 256 e3m2 tiles, k-steps split between two groups of four waves
constexpr int KSPLIT_THREADS = 512;
constexpr int KSPLIT_LDS = 4 * (128 + BN) * 96;
__global__ __launch_bounds__(KSPLIT_THREADS, 1) void k_gemm_w4a4_e3m2_ksplit(GemmArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    gemm_e3m2_ksplit(a, lds);
}

// int4 codes (two per byte, low nibble first) -> the tiled e3m2 layout.
// The 32 codes of unit u (k = 128 b + 32 u + e, e = 0..31) of row r form the
// 192-bit word sum_e code(q_e) << 6e, code(q) being q in e3m2 (sign, 3
// exponent bits of bias 3, 2 mantissa bits; every integer in -8..8 is exact).
// K-block b takes rows * 96 bytes at b * rows * 96: first the 64-byte heads
// of all rows (dwords 0-3 of unit u at 16-byte slot u ^ ((r >> 1) & 3) of the
// row's head), then the 32-byte tails (dwords 4-5 of unit u at 8-byte slot
// u ^ ((r >> 2) & 3)).  The GEMM moves a tile's k-step as consecutive
// kilobytes, and the slot swizzles make its LDS reads conflict-free.
// One thread per (b, r, u), u fastest.
__global__ __launch_bounds__(256) void k_pack_e3m2(const uint8_t *__restrict__ q4,
                                                   uint8_t *__restrict__ q6, int64_t rows,
                                                   int kb)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= rows * kb * 4)
        return;
    const int u = (int)(t & 3);
    const int64_t rb = t >> 2;
    const int64_t r = rb % rows;
    const int b = (int)(rb / rows);
    const uint4 in = *reinterpret_cast<const uint4 *>(q4 + r * ((int64_t)kb * 64) + (4 * b + u) * 16);
    const uint32_t w[4] = {in.x, in.y, in.z, in.w};
    uint32_t o[6];
    e3m2_unit(w, o);
    *reinterpret_cast<uint4 *>(q6 + e3m2_head(rows, r, b, u)) = make_uint4(o[0], o[1], o[2], o[3]);
    *reinterpret_cast<uint2 *>(q6 + e3m2_tail(rows, r, b, u)) = make_uint2(o[4], o[5]);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s, int bits)
{
    if (a.M == 0 || a.N == 0)
        return hipSuccess;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    const GemmPlan plan = plan_gemm(a.M, a.N, a.K, bits, cus, S);
    const int grid = plan.grid;
    if (plan.kernel == GemmKernel::K64) {
        hipError_t e = hipFuncSetAttribute((const void *)k_gemm_w4a4_k64,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
        if (e != hipSuccess)
            return e;
        hipLaunchKernelGGL(k_gemm_w4a4_k64, dim3((unsigned)grid), dim3(THREADS), LDS_BYTES, s, a);
        return hipGetLastError();
    }
    const bool ksplit = plan.kernel == GemmKernel::Ksplit;
    const bool m128 = plan.kernel == GemmKernel::Tile128;
    const void *fn;
    int lds_bytes, threads;
    if (ksplit) {
        fn = (const void *)k_gemm_w4a4_e3m2_ksplit;
        lds_bytes = KSPLIT_LDS;
        threads = KSPLIT_THREADS;
    } else if (m128) {
        fn = bits == 8 ? (const void *)k_gemm_w8a8_m128
             : bits == 6 ? (const void *)k_gemm_w4a4_e3m2_m128
                         : (const void *)k_gemm_w4a4_m128;
        lds_bytes = bits == 6 ? Ring<6, 128>::LDS : Ring<4, 128>::LDS;
        threads = Tile<128>::THREADS;
    } else {
        fn = bits == 8 ? (const void *)k_gemm_w8a8
             : bits == 6 ? (const void *)k_gemm_w4a4_e3m2
                         : (const void *)k_gemm_w4a4;
        lds_bytes = bits == 6 ? Ring<6>::LDS : Ring<4>::LDS;
        threads = Tile<256>::THREADS;
    }
    // more than 64 KB of dynamic LDS: raise the kernel's limit (per call, so
    // that every device the caller uses gets it; the call is host-side only)
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess)
        return e;
    GemmArgs args = a;
    void *params[] = {&args};
    e = hipLaunchKernel(fn, dim3((unsigned)grid), dim3((unsigned)threads), params,
                        (size_t)lds_bytes, s);
    if (e != hipSuccess)
        return e;
    return hipGetLastError();
}

hipError_t launch_pack_e3m2(const uint8_t *q4, uint8_t *q6, int64_t rows, int k, hipStream_t s)
{
    const int kb = k / 128;
    const int64_t threads = rows * kb * 4;
    if (threads == 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_pack_e3m2, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, q4,
                       q6, rows, kb);
    return hipGetLastError();
}

}  // namespace quarot
