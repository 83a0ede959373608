// Host build of the library's bit-level encoders (the same source the GPU
// kernels compile), checked over all their inputs against references
// written here from the definitions:
//  - e3m2 (sign, 3 exponent bits of bias 3, 2 mantissa bits, subnormals at
//    exponent field 0): the code of every int4 value and its placement in a
//    192-bit unit (code e at bits 6e), for every value at every position of
//    a unit and for random units (e3m2_of_bits, e3m2_lut4,
//    e3m2_of_nibbles8, e3m2_unit);
//  - the tiled layout's head/tail slots: every (row, unit) of a block maps
//    to distinct bytes that cover the block exactly (e3m2_head, e3m2_tail);
//  - the signed base-64 digits of an fp16 value: for all 65536 encodings of
//    finite values, sum_k digit_k 64^k = value * 2^24 exactly with digits in
//    [-63, 63], and the 4-value plane transpose (f16_planes, f16x4_planes).
// Prints "ok" and exits 0, or names the first failure and exits 1.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "../../paper_2404_00456_amd/csrc/common.hpp"

using namespace quarot;

static double e3m2_value(uint32_t c)
{
    const double s = (c & 0x20u) ? -1.0 : 1.0;
    const uint32_t e = (c >> 2) & 7u, m = c & 3u;
    if (e == 0)
        return s * std::ldexp((double)m / 4.0, -2);
    return s * std::ldexp(1.0 + (double)m / 4.0, (int)e - 3);
}

static double f16_value(uint32_t h)
{
    const double s = (h & 0x8000u) ? -1.0 : 1.0;
    const int e = (h >> 10) & 31;
    const int m = h & 1023;
    if (e == 0)
        return s * std::ldexp((double)m, -24);
    return s * std::ldexp(1024.0 + m, e - 25);
}

static int fail(const char *what, long a, long b)
{
    std::printf("FAIL %s (%ld, %ld)\n", what, a, b);
    return 1;
}

int main()
{
    // e3m2 code of every integer -8..8 from its binary32 encoding
    for (int q = -8; q <= 8; ++q) {
        float f = (float)q;
        uint32_t b;
        std::memcpy(&b, &f, 4);
        const uint32_t c = e3m2_of_bits(b);
        if (c > 63 || e3m2_value(c) != (double)q || (q == 0 && c != 0))
            return fail("e3m2_of_bits", q, c);
    }
    // units: every nibble value at every position, then random units
    auto check_unit = [&](const uint32_t (&w)[4]) -> bool {
        uint32_t o[6];
        e3m2_unit(w, o);
        for (int e = 0; e < 32; ++e) {
            const int nib = (w[e / 8] >> (4 * (e % 8))) & 15;
            const int q = nib >= 8 ? nib - 16 : nib;
            const int bit = 6 * e;
            uint64_t word = o[bit / 32] | ((bit / 32 + 1 < 6) ? (uint64_t)o[bit / 32 + 1] << 32 : 0);
            const uint32_t c = (uint32_t)(word >> (bit % 32)) & 63u;
            if (e3m2_value(c) != (double)q)
                return false;
        }
        return true;
    };
    for (int pos = 0; pos < 32; ++pos)
        for (int v = 0; v < 16; ++v) {
            uint32_t w[4] = {0x13579BDFu, 0x02468ACEu, 0xFEDCBA98u, 0x76543210u};
            w[pos / 8] = (w[pos / 8] & ~(15u << (4 * (pos % 8)))) | ((uint32_t)v << (4 * (pos % 8)));
            if (!check_unit(w))
                return fail("e3m2_unit position/value", pos, v);
        }
    std::mt19937_64 rng(1);
    for (int t = 0; t < 200000; ++t) {
        const uint32_t w[4] = {(uint32_t)rng(), (uint32_t)rng(), (uint32_t)rng(), (uint32_t)rng()};
        if (!check_unit(w))
            return fail("e3m2_unit random", t, 0);
    }
    // tiled layout: the heads and tails of every (row, unit) of a block
    // partition the block's rows * 96 bytes
    for (int64_t rows : {1, 2, 3, 16, 37, 256, 1000}) {
        std::vector<int> hit((size_t)rows * 96, 0);
        for (int64_t r = 0; r < rows; ++r)
            for (int u = 0; u < 4; ++u) {
                const int64_t h = e3m2_head(rows, r, 0, u), t = e3m2_tail(rows, r, 0, u);
                for (int i = 0; i < 16; ++i)
                    hit[(size_t)(h + i)]++;
                for (int i = 0; i < 8; ++i)
                    hit[(size_t)(t + i)]++;
                if (e3m2_head(rows, r, 3, u) != h + 3 * rows * 96)
                    return fail("e3m2_head block stride", rows, r);
            }
        for (size_t i = 0; i < hit.size(); ++i)
            if (hit[i] != 1)
                return fail("e3m2 layout coverage", rows, (long)i);
    }
    // signed base-64 digits of every finite fp16 value
    for (uint32_t h = 0; h < 65536; ++h) {
        if (((h >> 10) & 31) == 31)
            continue;
        const uint64_t p = f16_planes(h);
        long double sum = 0;
        for (int k = 0; k < 8; ++k) {
            const int d = (int8_t)(uint8_t)(p >> (8 * k));
            if (d < -63 || d > 63 || (k == 7 && d != 0))
                return fail("f16_planes digit range", h, k);
            sum += (long double)d * std::pow(64.0L, k);
        }
        if (sum != (long double)f16_value(h) * 16777216.0L)
            return fail("f16_planes value", h, 0);
    }
    for (int t = 0; t < 200000; ++t) {
        uint32_t h[4];
        for (int i = 0; i < 4; ++i) {
            do
                h[i] = (uint32_t)rng() & 0xFFFFu;
            while (((h[i] >> 10) & 31) == 31);
        }
        uint32_t w[7];
        f16x4_planes(make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16)), w);
        for (int i = 0; i < 4; ++i)
            for (int k = 0; k < 7; ++k)
                if (((w[k] >> (8 * i)) & 0xFFu) != ((f16_planes(h[i]) >> (8 * k)) & 0xFFu))
                    return fail("f16x4_planes transpose", t, 7 * i + k);
    }
    std::printf("ok\n");
    return 0;
}
