// Checks nuna::udiv (fastdiv.h) against the hardware quotient: every divisor
// up to 4096 with the numerators below 2^16 and the 40001 just below 2^31, then
// random divisors of every magnitude with random numerators, exact multiples
// and their neighbours.  Prints the count of mismatches; exit status 1 if any.
#include <cstdint>
#include <cstdio>
#include <random>

#include "fastdiv.h"

int main() {
    long long checked = 0, bad = 0;
    auto check = [&](uint32_t n, uint32_t d, const nuna::Magic& g) {
        ++checked;
        if (nuna::udiv(n, g) != n / d) {
            if (++bad <= 10) std::printf("mismatch: %u / %u\n", n, d);
        }
    };
    for (uint32_t d = 1; d <= 4096; ++d) {
        const nuna::Magic g = nuna::make_magic(d);
        for (uint32_t n = 0; n < (1u << 16); ++n) check(n, d, g);
        for (uint32_t n = 0x7FFFFFFFu - 40000; n <= 0x7FFFFFFFu; ++n) check(n, d, g);
    }
    std::mt19937_64 r(20260601);
    for (int i = 0; i < 4000000; ++i) {
        const uint32_t d = 1 + static_cast<uint32_t>((r() & 0x7FFFFFFFu) >> (r() % 31));
        const nuna::Magic g = nuna::make_magic(d);
        check(static_cast<uint32_t>(r() & 0x7FFFFFFFu), d, g);
        const uint64_t q = (r() & 0x7FFFFFFFu) / d;
        for (int o = -1; o <= 1; ++o) {
            const int64_t n = static_cast<int64_t>(q * d) + o;
            if (n >= 0 && n <= 0x7FFFFFFF) check(static_cast<uint32_t>(n), d, g);
        }
    }
    std::printf("fastdiv: %lld quotients checked, %lld mismatches\n", checked, bad);
    return bad != 0;
}
