// fastdiv.h -- division by a divisor fixed for a whole launch.
//
// The host turns each divisor d into a multiplier and a shift once; the kernel
// then divides with a multiply-high, an add and a shift instead of the ~25
// dependent instructions of a general 32-bit division (Granlund and
// Montgomery, "Division by invariant integers using multiplication", PLDI
// 1994, round-up method). With l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, which fits 32 bits, every n < 2^31 has
//   n / d = (mulhi(n, m) + n) >> l,
// and the add cannot overflow because mulhi(n, m) < n.
#pragma once

#include <stdint.h>

struct FastDiv {
    uint32_t mul;
    uint32_t shift;
    uint32_t d;
};

// 1 <= d < 2^31.
constexpr FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while (l < 31 && (1u << l) < d) ++l;
    const uint64_t m = ((((uint64_t)1 << l) - d) << 32) / d + 1;
    return FastDiv{(uint32_t)m, l, d};
}

// n / d for 0 <= n < 2^31.
constexpr uint32_t fast_div(uint32_t n, FastDiv f)
{
    return (uint32_t)((((uint64_t)n * f.mul) >> 32) + n) >> f.shift;
}
