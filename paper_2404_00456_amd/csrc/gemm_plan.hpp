// Host-side choice of the integer GEMM kernel and its grid from the
// problem's shape and the device's CU count.  Plain C++ with no HIP, so the
// rule builds and is checked on any host.
#pragma once

#include <cstdint>

namespace quarot {
namespace gemm {

enum class GemmKernel {
    K64,      // int4 codes with K not a multiple of 128: one 256 x 256 tile per block
    Tile256,  // persistent, 256 x 256 block tiles
    Tile128,  // persistent, 128 x 256 block tiles, one wave per SIMD
    Ksplit,   // e3m2 only: 128 x 256 tiles, k-steps split between two wave groups
};

struct GemmPlan {
    GemmKernel kernel;
    int grid;  // blocks
};

// bits: 4 (int4 codes widened to int8), 6 (int4 codes as e3m2 numbers) or
// 8 (int8 codes); cus: the device's compute units; stages: the depth of the
// persistent kernels' LDS ring.  M, N > 0; the caller returns before
// planning an empty output.
inline GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int bits, int cus, int stages)
{
    constexpr int64_t TILE = 256;
    if (bits == 4 && K % 128 != 0)
        return {GemmKernel::K64, (int)(((M + TILE - 1) / TILE) * ((N + TILE - 1) / TILE))};
    const int64_t ksteps = bits == 8 ? K / 64 : K / 128;
    // 128-row block tiles when that takes less time over the CUs: with one
    // wave per SIMD a 128 x 256 tile takes about 0.9 of a 256 x 256 tile's
    // time (measured on the 7B down-projection shape: 74.6 against 81.8 us
    // for one round each), so only grids that leave CUs idle gain (2048 x
    // 4096 outputs: 128 large tiles for 256 CUs), not the 16384-token ones.
    const int64_t TN = (N + TILE - 1) / TILE;
    const int64_t t256 = ((M + 255) / 256) * TN, t128 = ((M + 127) / 128) * TN;
    const int64_t r256 = (t256 + cus - 1) / cus, r128 = (t128 + cus - 1) / cus;
    // e3m2 codes with K a multiple of 256: the 128-row tiles with the
    // k-steps split between two wave groups, which take about KSPLIT_COST %
    // of a 256 x 256 tile's time
    constexpr int64_t KSPLIT_COST = 70;
    const bool ksplit =
        bits == 6 && K % 256 == 0 && K >= 512 && M > 128 && r128 * KSPLIT_COST < r256 * 100;
    const bool m128 = ksplit || (ksteps >= stages && M > 128 && r128 * 90 < r256 * 100);
    const int64_t tiles = m128 ? t128 : t256;
    // persistent: one block per CU, or fewer for small problems (the LDS
    // ring allows one resident block per CU); with fewer than `stages`
    // k-steps, one tile per block.  A grid of whole groups of eight when the
    // tiles come in such groups, so that each XCD takes the same share.
    int64_t grid = (tiles < cus || ksteps < stages) ? tiles : cus;
    if (grid >= 8 && tiles % 8 == 0)
        grid -= grid % 8;
    return {ksplit ? GemmKernel::Ksplit : m128 ? GemmKernel::Tile128 : GemmKernel::Tile256,
            (int)grid};
}

}  // namespace gemm
}  // namespace quarot
