// stream.hpp -- the seeded challenge stream of a context (ra_ctx_create) and
// of the seeded verifier (ra_verify): xorshift64 with shifts (13, 7, 17)
// (Marsaglia, "Xorshift RNGs", J. Stat. Softw. 8(14), 2003) from a nonzero
// 64-bit state; each challenge is the next output reduced modulo
// p = 2^61 - 1.  Host code.
#pragma once
#include <cstdint>

namespace ra {

struct ChallengeStream {
    uint64_t x;
    explicit ChallengeStream(uint64_t seed) : x(seed) {}
    uint64_t next()
    {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        const uint64_t p = 0x1FFFFFFFFFFFFFFFull;
        const uint64_t r = (x & p) + (x >> 61);  // 2^61 = 1 mod p; r < 2^61 + 8
        return r >= p ? r - p : r;
    }
};

}  // namespace ra
