// Checks smol_magic.h's division by multiplication against integer division:
// every divisor 1 .. 2^16 with numerators at and around its multiples and at
// the ends of the range, then large divisors with seeded numerators. Prints
// the number of checks, or the first failure and exits 1.
#include <cstdio>
#include <random>

#include "smol_magic.h"

static long long checks = 0;

static bool check(uint32_t n, uint32_t d, uint32_t m, uint32_t s)
{
    ++checks;
    const uint32_t q = smol::magic_div(n, m, s);
    if (q != n / d) {
        std::printf("FAIL n=%u d=%u m=%u s=%u: %u != %u\n", n, d, m, s, q, n / d);
        return false;
    }
    return true;
}

int main()
{
    const uint32_t top = 0x7fffffffu;  // numerators are below 2^31
    std::mt19937_64 rng(13005);
    for (uint32_t d = 1; d <= 65536; ++d) {
        uint32_t m, s;
        smol::magic_divisor(d, &m, &s);
        const uint32_t k = top / d;
        for (uint32_t n : {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, top, top - 1,
                           k * d, k * d - 1, (k / 2) * d, (k / 2) * d - 1})
            if (n <= top && !check(n, d, m, s))
                return 1;
        for (int t = 0; t < 16; ++t)
            if (!check((uint32_t)(rng() & top), d, m, s))
                return 1;
    }
    for (int t = 0; t < 200000; ++t) {
        const uint32_t d = 1 + (uint32_t)(rng() % top);
        uint32_t m, s;
        smol::magic_divisor(d, &m, &s);
        const uint32_t n = (uint32_t)(rng() & top);
        if (!check(n, d, m, s) || !check(top, d, m, s) || !check(d - 1, d, m, s) ||
            !check((top / d) * d, d, m, s))
            return 1;
    }
    std::printf("checks %lld\n", checks);
    return 0;
}
