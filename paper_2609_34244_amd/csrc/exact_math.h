// Exact integer helpers shared by the host and the gfx950 kernels of the
// pricing library.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
#define HEDDLE_HD __host__ __device__ __forceinline__
#else
#define HEDDLE_HD static inline
#endif

namespace heddle {

// ceil(x * a / d) for x < 2^51, a < 2^28, 1 <= d < 2^50; the result is below
// 2^62. gfx950 has no integer divider and a 128-bit division expands to a
// bit-serial loop, so the quotient is estimated in fp64 and corrected exactly.
// When x * a + d - 1 < 2^53 one fp64 division and one correction step do;
// otherwise:
// the first estimate is within 2^11 of the true quotient (relative error of
// the fp64 operands and division is below 2^-51 and the quotient below 2^62),
// which leaves a remainder |r| < 2^12 d < 2^62 that fits int64; the second
// estimate r / d is then off by at most one, fixed by one exact step.
HEDDLE_HD uint64_t ceil_muldiv(uint64_t x, uint64_t a, uint64_t d)
{
    const unsigned __int128 n = (unsigned __int128)x * a + (d - 1);     // ceil -> floor
    if ((uint64_t)(n >> 53) == 0) {
        // n and d are exact doubles; the correctly rounded quotient lies within
        // one of floor(n / d) (within half of n / d, and n / d < 2^53), and one
        // exact step on the remainder r = n - q d, |r| < 2d, corrects it
        const uint64_t nl = (uint64_t)n;
        int64_t q = (int64_t)((double)nl / (double)d);
        const int64_t r = (int64_t)(nl - (uint64_t)q * d);
        if (r < 0) q -= 1;
        else if (r >= (int64_t)d) q += 1;
        return (uint64_t)q;
    }
    const double dd = (double)d;
    const double nd = (double)(uint64_t)(n >> 64) * 18446744073709551616.0 + (double)(uint64_t)n;
    int64_t q = (int64_t)(nd / dd);
    int64_t r = (int64_t)(uint64_t)(n - (unsigned __int128)(uint64_t)q * d);   // |r| < 2^62: low word is exact
    q += (int64_t)__builtin_floor((double)r / dd);
    r = (int64_t)(uint64_t)(n - (unsigned __int128)(uint64_t)q * d);
    if (r < 0) q -= 1;
    else if (r >= (int64_t)d) q += 1;
    return (uint64_t)q;
}

// Ring all-reduce of b bytes over n ranks at bw MB/s, in ns:
// ceil(2 (n-1) b * 1000 / (n bw)); zero for one rank.
HEDDLE_HD int64_t allreduce_ns(int64_t b, int64_t n, int64_t bw)
{
    if (n <= 1 || b == 0) return 0;
    return (int64_t)ceil_muldiv((uint64_t)b, (uint64_t)(2 * (n - 1)) * 1000u, (uint64_t)(n * bw));
}

}  // namespace heddle
