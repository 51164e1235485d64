// fastdiv.h -- division by a divisor known only at run time, as a multiply
// and a shift.
//
// GPU code has no integer divide instruction: n / d with a run-time d expands
// to a long sequence of floating-point reciprocal and correction steps.  Where
// every workgroup divides many values by the same divisor (the routed MoE
// dispatch: expert to rank, item to token, token to source rank), the host
// computes once, for d >= 1,
//     l = ceil(log2 d),  m = ceil(2^(31 + l) / d)   (m < 2^32),
// and then n / d = (m * n) >> (31 + l) for every 0 <= n < 2^31 (Granlund and
// Montgomery, "Division by invariant integers using multiplication", PLDI
// 1994, Thm. 4.2 with N = 31): m * d lies in [2^(31+l), 2^(31+l) + 2^l].
// tests/c/fastdiv_check.cpp checks it against the hardware quotient.
#ifndef NUNA_FASTDIV_H
#define NUNA_FASTDIV_H

#include <cstdint>

#ifndef NUNA_HD
#if defined(__HIPCC__)
#define NUNA_HD __host__ __device__
#else
#define NUNA_HD
#endif
#endif

namespace nuna {

struct Magic {
    uint32_t m;
    int32_t sh;
};

// Host: the constants for divisor d (d = 0 is taken as 1).
inline Magic make_magic(uint32_t d) {
    if (d == 0) d = 1;
    int l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    const uint64_t num = uint64_t(1) << (31 + l);
    return {static_cast<uint32_t>((num + d - 1) / d), 31 + l};
}

// n / d for 0 <= n < 2^31.
NUNA_HD inline uint32_t udiv(uint32_t n, const Magic& g) {
    return static_cast<uint32_t>((static_cast<uint64_t>(g.m) * n) >> g.sh);
}

}  // namespace nuna

#endif
