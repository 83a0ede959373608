// The integer GEMM launcher's kernel and grid choice (csrc/gemm_plan.hpp),
// built for the host: the Llama-2 70B and 7B projection shapes on each code
// width, and the boundaries of every branch of the rule.
#include <cstdio>

#include "gemm_plan.hpp"

using quarot::gemm::GemmKernel;
using quarot::gemm::plan_gemm;

static const char *name(GemmKernel k)
{
    switch (k) {
    case GemmKernel::K64: return "K64";
    case GemmKernel::Tile256: return "Tile256";
    case GemmKernel::Tile128: return "Tile128";
    case GemmKernel::Ksplit: return "Ksplit";
    }
    return "?";
}

struct Case {
    long long M, N, K;
    int bits, cus;
    GemmKernel kernel;
    int grid;
};

int main()
{
    const Case cases[] = {
        // Llama-2 70B FFN at 16384 tokens: 7168 and 2048 large tiles, one block per CU
        {16384, 28672, 8192, 6, 256, GemmKernel::Tile256, 256},
        {16384, 8192, 28672, 6, 256, GemmKernel::Tile256, 256},
        {16384, 28672, 8192, 4, 256, GemmKernel::Tile256, 256},
        {16384, 28672, 8192, 8, 256, GemmKernel::Tile256, 256},
        // Llama-2 7B at 2048 tokens: up keeps 344 large tiles in two rounds;
        // down (128 large tiles) takes 256 128-row tiles, split k on e3m2
        {2048, 11008, 4096, 6, 256, GemmKernel::Tile256, 256},
        {2048, 11008, 4096, 4, 256, GemmKernel::Tile256, 256},
        {2048, 4096, 11008, 6, 256, GemmKernel::Ksplit, 256},
        {2048, 4096, 11008, 4, 256, GemmKernel::Tile128, 256},
        {2048, 4096, 11008, 8, 256, GemmKernel::Tile128, 256},
        // int4 codes with K not a multiple of 128: one tile per block
        {300, 520, 100, 4, 256, GemmKernel::K64, 6},
        // split k needs M > 128, K a multiple of 256 and at least 512
        {128, 4096, 4096, 6, 256, GemmKernel::Tile256, 16},
        {129, 4096, 4096, 6, 256, GemmKernel::Ksplit, 32},
        {129, 300, 512, 6, 256, GemmKernel::Ksplit, 4},
        {2048, 8448, 384, 6, 256, GemmKernel::Tile256, 256},
        // fewer k-steps than ring stages: one tile per block, every tile a block
        {2048, 8448, 256, 6, 256, GemmKernel::Tile256, 264},
        {16, 256, 128, 6, 256, GemmKernel::Tile256, 1},
        // 387 small tiles, two rounds either way: split k, 256 blocks
        {384, 33000, 512, 6, 256, GemmKernel::Ksplit, 256},
        // other CU counts: grids of whole groups of eight when the tiles are
        {4096, 4096, 4096, 6, 100, GemmKernel::Tile256, 96},
        {2048, 4096, 11008, 6, 304, GemmKernel::Ksplit, 256},
        {1000, 36, 768, 6, 256, GemmKernel::Ksplit, 8},
    };
    int failures = 0;
    for (const Case &c : cases) {
        const auto p = plan_gemm(c.M, c.N, c.K, c.bits, c.cus, 3);
        if (p.kernel != c.kernel || p.grid != c.grid) {
            std::printf("FAIL M=%lld N=%lld K=%lld bits=%d cus=%d: %s grid %d, want %s grid %d\n",
                        c.M, c.N, c.K, c.bits, c.cus, name(p.kernel), p.grid, name(c.kernel),
                        c.grid);
            ++failures;
        }
    }
    if (failures)
        return 1;
    std::printf("ok\n");
    return 0;
}
