// qfastdiv.h -- division by a run-time invariant divisor (host + device).
#pragma once

#include <stdint.h>

namespace ql {

// ---------------------------------------------------------------------------
// Division by a run-time constant via a precomputed multiplier (the
// round-up method of Granlund & Montgomery, "Division by invariant integers
// using multiplication", PLDI 1994): q = (mulhi(n, m) + n) >> s with
// s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1.  Exact for every 32-bit n (the sum is formed in 64 bits).
// ---------------------------------------------------------------------------
struct FastDiv {
    uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t s = 0;
    while ((1ull << s) < d) ++s;
    f.s = s;
    f.m = (uint32_t)((((1ull << s) - d) << 32) / d + 1);
    return f;
}

// Host-side evaluation of the same formula (used by the host code and its tests).
inline uint32_t fdiv_host(uint32_t n, const FastDiv &f) {
    return (uint32_t)(((((uint64_t)n * f.m) >> 32) + (uint64_t)n) >> f.s);
}

}  // namespace ql
