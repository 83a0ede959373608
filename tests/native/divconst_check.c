/* Division by a small integer constant d without a division instruction:
 * r = RN(1/d), q0 = RN(x r), e = x - q0 d (exact by one fma),
 * q = RN(q0 + e r) (one fma).  Counts the positive finite binary32 x whose
 * q differs from the IEEE quotient RN(x / d); negative x mirror positive
 * ones (every step is odd in x under round-to-nearest-even). */
#include <math.h>
#include <stdint.h>
#include <string.h>

long divconst_check(float d, uint32_t first, uint32_t last)
{
    const float r = 1.0f / d;
    long bad = 0;
#pragma omp parallel for schedule(static) reduction(+ : bad)
    for (int64_t bb = first; bb <= (int64_t)last; bb++) {
        const uint32_t b = (uint32_t)bb;
        float x;
        memcpy(&x, &b, 4);
        const float q0 = x * r;
        const float e = fmaf(-q0, d, x);
        const float q = fmaf(e, r, q0);
        const float ref = x / d;
        if (memcmp(&q, &ref, 4) != 0)
            bad++;
    }
    return bad;
}
