/* Exhaustive check of the binary32 division by the total mass used by the
 * step kernels: q = x * RN(1/M); r = fma(-q, M, x); q' = fma(r, RN(1/M), q)
 * against the correctly rounded x / M, for every finite binary32 x
 * (M = 0.1f + 1.0f).  Prints the number of mismatches and the largest |x|
 * with one (0 if none).  Built and run by tests/test_division_by_mass.py. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

int main(void) {
    const float m = 0.1f + 1.0f;
    const float inv = 1.0f / m;
    long mismatches = 0;
    float worst = 0.0f;
#pragma omp parallel for reduction(+ : mismatches) reduction(max : worst) schedule(static)
    for (int64_t u = 0; u < 0x100000000LL; ++u) {
        const uint32_t bits = (uint32_t)u;
        float x;
        memcpy(&x, &bits, 4);
        if (!isfinite(x)) continue;
        const float ref = x / m;
        const float q = x * inv;
        const float r = fmaf(-q, m, x);
        const float q2 = fmaf(r, inv, q);
        if (memcmp(&ref, &q2, 4) != 0) {
            ++mismatches;
            if (fabsf(x) > worst) worst = fabsf(x);
        }
    }
    printf("%ld %a\n", mismatches, (double)worst);
    return 0;
}
