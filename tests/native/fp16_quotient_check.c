/*
 * Exhaustive check, over every pair of binary16 operands, that the quotient
 * the quantize kernel forms,
 *     y  = RN(1 / s)                  (one IEEE division per group)
 *     q  = RN(v * y + 0)              (fused; RN(v * y) up to the sign of a zero)
 *     r  = RN(v - q * s)              (fused multiply-add: q * s exact)
 *     q' = RN(q + r * y)              (fused multiply-add)
 * equals the IEEE binary32 quotient RN(v / s) for every finite fp16 v and
 * every finite positive fp16 s (the whole input domain: weights and scales
 * are fp16 values).  Equality is compared as values (-0 == +0; both give
 * the same code).  Prints the number of pairs and of mismatches.
 *
 * Build: gcc -O2 -std=c11 -fno-fast-math -ffp-contract=off -mfma -fopenmp
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>

static float half_to_float(uint16_t h)
{
    int sign = h >> 15, e = (h >> 10) & 31, f = h & 1023;
    float v = (e == 0) ? ldexpf((float)f, -24) : ldexpf((float)(1024 + f), e - 25);
    return sign ? -v : v;
}

int main(void)
{
    long long pairs = 0, bad = 0;
#pragma omp parallel for reduction(+ : pairs, bad) schedule(dynamic, 64)
    for (int sb = 1; sb < 0x7C00; ++sb) {
        const float s = half_to_float((uint16_t)sb);
        const float y = 1.0f / s;
        for (int vb = 0; vb < 0x10000; ++vb) {
            if (((vb >> 10) & 31) == 31)
                continue; /* inf / NaN weights are outside the domain */
            const float v = half_to_float((uint16_t)vb);
            const float q = fmaf(v, y, 0.0f); /* RN(v * y) up to the sign of a zero */
            const float r = fmaf(-q, s, v);
            const float q2 = fmaf(r, y, q);
            pairs++;
            if (!(q2 == v / s))
                bad++;
        }
    }
    printf("%lld %lld\n", pairs, bad);
    return 0;
}
