/* Checks, for a divisor b and every sampled fp32 a whose quotient is a normal
 * number, that the quotient formed from the correctly rounded reciprocal
 * y = RN(1/b) with one FMA correction,
 *     q0 = RN(a * y);  q = RN(q0 + RN(a - b*q0) * y),
 * equals the IEEE quotient RN(a / b). The kernels normalise with that
 * sequence; this program is the CPU-side evidence that it is exact.
 * Usage: div_identity STRIDE b1 [b2 ...]   (mantissa sampling stride) */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int main(int argc, char **argv)
{
    if (argc < 3)
        return 2;
    uint32_t stride = (uint32_t)atoi(argv[1]);
    long long bad = 0, n = 0;
    for (int k = 2; k < argc; ++k) {
        volatile float b = (float)atof(argv[k]);
        float y = 1.0f / b;
        /* |a| in [2^-100, 2^10): covers every v - mean the kernels produce */
        for (uint32_t e = 27; e <= 136; ++e)
            for (uint32_t m = (e * 7919u) % stride; m < (1u << 23); m += stride)
                for (uint32_t s = 0; s < 2; ++s) {
                    uint32_t u = (s << 31) | (e << 23) | m;
                    float a;
                    memcpy(&a, &u, 4);
                    float q = a / b;
                    float q0 = a * y;
                    float q1 = fmaf(fmaf(-b, q0, a), y, q0);
                    ++n;
                    if (memcmp(&q, &q1, 4) != 0) {
                        if (bad < 5)
                            printf("mismatch b=%a a=%a q=%a q1=%a\n", b, a, q, q1);
                        ++bad;
                    }
                }
    }
    printf("%lld mismatches of %lld\n", bad, n);
    return bad != 0;
}
