// smol_magic.h -- division by a fixed divisor as a multiplication (host
// side): the block-decoding kernel maps job indices to blocks with the
// multipliers computed here (JpegRun in smol_internal.h).
#pragma once

#include <stdint.h>

namespace smol {

// m = ceil(2^s / d), s = 31 + ceil(log2 d), for 1 <= d < 2^31: then
// floor(n / d) = floor(n m / 2^s) for every 0 <= n < 2^31. (m = (2^s + e) / d
// with 0 <= e < d, so n m / 2^s exceeds n / d by e n / (d 2^s) < 2^-ceil(log2 d)
// <= 1 / d, which cannot carry n / d past the next integer.) m < 2^32.
inline void magic_divisor(uint32_t d, uint32_t *m, uint32_t *s)
{
    int l = 0;
    while (((uint64_t)1 << l) < d)
        ++l;
    *s = (uint32_t)(31 + l);
    *m = (uint32_t)((((uint64_t)1 << (31 + l)) + d - 1) / d);
}

// floor(n / d) from magic_divisor's m and s, as the kernel evaluates it.
inline uint32_t magic_div(uint32_t n, uint32_t m, uint32_t s)
{
    return (uint32_t)(((uint64_t)n * m) >> s);
}

}  // namespace smol
