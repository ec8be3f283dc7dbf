// Checks fast_div against the hardware division: every dividend below 3000
// and multiples of d plus or minus one for d = 1..70000, random dividends
// below 2^31 for those and for random divisors below 2^31, and divisors next
// to every power of two. Exit status 1 on any mismatch.
#include "fastdiv.h"

#include <cstdio>
#include <random>

int main()
{
    std::mt19937_64 g(1);
    long bad = 0, checks = 0;
    auto check = [&](uint32_t n, uint32_t d, FastDiv f) {
        ++checks;
        if (fast_div(n, f) != n / d && bad++ < 10) std::printf("mismatch: n=%u d=%u\n", n, d);
    };
    for (uint32_t d = 1; d <= 70000; ++d) {
        const FastDiv f = make_fastdiv(d);
        for (uint32_t n = 0; n < 3000; ++n) check(n, d, f);
        for (int i = 0; i < 200; ++i) check((uint32_t)(g() & 0x7fffffff), d, f);
        for (uint64_t q = 1; q < 40; ++q)
            for (int e = -1; e <= 1; ++e)
                if (q * d + e < 0x80000000ull) check((uint32_t)(q * d + e), d, f);
        check(0x7fffffffu, d, f);
    }
    for (int i = 0; i < 2000000; ++i) {
        const uint32_t d = (uint32_t)(g() % 0x7fffffff) + 1;
        const FastDiv f = make_fastdiv(d);
        check((uint32_t)(g() & 0x7fffffff), d, f);
        check(0x7fffffffu, d, f);
        check(d - 1, d, f);
        check(d, d, f);
    }
    for (uint32_t l = 0; l < 31; ++l)
        for (int e = -1; e <= 1; ++e) {
            const int64_t d = ((int64_t)1 << l) + e;
            if (d < 1 || d >= 0x80000000ll) continue;
            const FastDiv f = make_fastdiv((uint32_t)d);
            for (int i = 0; i < 20000; ++i) check((uint32_t)(g() & 0x7fffffff), (uint32_t)d, f);
            check(0x7fffffffu, (uint32_t)d, f);
        }
    std::printf("%ld checks, %ld mismatches\n", checks, bad);
    return bad != 0;
}
