/*
 * Test helper: checks that Markstein's correction,
 *   r = RN(1/s), q0 = RN(y r), e = fma(-q0, s, y), q = fma(e, r, q0),
 * yields the same int4/uint4 code as IEEE division, clamp(rint(RN(y/s))),
 * for every positive finite binary16 divisor s (the quantizers' stored
 * scales) and many numerators: uniform quotients, quotients within a few
 * ulps of half-integers and integers, and arbitrary binary32 values.
 * Returns the number of code mismatches and counts the quotient
 * mismatches and the largest |q| among them.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static float half_to_float(uint16_t h)
{
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16, e = (h >> 10) & 31u, m = h & 1023u, b;
    float f;
    if (!e) {
        f = (float)m * 5.9604644775390625e-8f;
        return sign ? -f : f;
    }
    b = sign | ((e - 15u + 127u) << 23) | (m << 13);
    memcpy(&f, &b, 4);
    return f;
}

long markstein_check(int samples, long *quot_mismatch, double *max_bad_q)
{
    long bad_code = 0, bad_q = 0;
    double worst = 0.0;
    for (int h = 1; h < 0x7C00; h++) {
        uint64_t st = 0x9E3779B97F4A7C15ull * (uint64_t)(h + 1);
        const float s = half_to_float((uint16_t)h), r = 1.0f / s;
        for (int t = 0; t < samples; t++) {
            st ^= st << 13;
            st ^= st >> 7;
            st ^= st << 17;
            float y;
            uint32_t b;
            int k = (int)(st % 17) - 8, jit = (int)((st >> 20) % 9) - 4;
            switch (t & 3) {
            case 0:
                y = (((float)(st >> 40) / 16777216.0f) * 18.0f - 9.0f) * s;
                break;
            case 1:
                y = ((float)k + 0.5f) * s;
                memcpy(&b, &y, 4);
                b += jit;
                memcpy(&y, &b, 4);
                break;
            case 2:
                y = (float)k * s;
                memcpy(&b, &y, 4);
                b += jit;
                memcpy(&y, &b, 4);
                break;
            default:
                b = (uint32_t)(st >> 32) & 0x7FFFFFFFu;
                if (((b >> 23) & 255u) == 255u)
                    b ^= 0x40000000u;
                memcpy(&y, &b, 4);
                if (st & 1)
                    y = -y;
            }
            if (!isfinite(y))
                continue;
            const float q = y / s;
            if (!isfinite(q))
                continue;
            const float q0 = y * r, e = fmaf(-q0, s, y), q1 = fmaf(e, r, q0);
            if (memcmp(&q, &q1, 4) != 0) {
                bad_q++;
                if (fabs(q) > worst)
                    worst = fabs(q);
            }
            float c1 = fminf(fmaxf(rintf(q), -8.0f), 7.0f), c2 = fminf(fmaxf(rintf(q1), -8.0f), 7.0f);
            float u1 = fminf(fmaxf(rintf(q), 0.0f), 15.0f), u2 = fminf(fmaxf(rintf(q1), 0.0f), 15.0f);
            if (c1 != c2 || u1 != u2)
                bad_code++;
        }
    }
    *quot_mismatch = bad_q;
    *max_bad_q = worst;
    return bad_code;
}
