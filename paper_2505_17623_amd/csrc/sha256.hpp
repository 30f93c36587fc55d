// sha256.hpp -- SHA-256 (FIPS 180-4) for the Fiat-Shamir transcript, on the
// host (the verifier) and on the device (the prover's transcript kernels and
// the Merkle root of the witness tables).
//
// The constants are computed at compile time from their definition: the
// first 32 bits of the fractional parts of the square roots of the first 8
// primes (initial hash value) and of the cube roots of the first 64 primes
// (round constants), by exact integer roots.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sha {

struct Consts {
    uint32_t h[8];
    uint32_t k[64];
};

constexpr unsigned __int128 int_root(unsigned __int128 v, int e)
{
    unsigned __int128 lo = 0, hi = (unsigned __int128)1 << (e == 2 ? 64 : 43);
    while (lo < hi) {
        const unsigned __int128 mid = lo + (hi - lo + 1) / 2;
        unsigned __int128 p = mid * mid;
        if (e == 3) p *= mid;
        if (p <= v) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

constexpr Consts make_consts()
{
    Consts c{};
    int n = 0;
    for (int x = 2; n < 64; x++) {
        bool prime = true;
        for (int d = 2; d * d <= x; d++)
            if (x % d == 0) prime = false;
        if (!prime) continue;
        if (n < 8) c.h[n] = (uint32_t)int_root((unsigned __int128)x << 64, 2);
        c.k[n] = (uint32_t)int_root((unsigned __int128)x << 96, 3);
        n++;
    }
    return c;
}

inline constexpr Consts kConsts = make_consts();

__host__ __device__ inline uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

// One compression of the 16 big-endian words w of a block into st.
__host__ __device__ inline void compress(uint32_t st[8], const uint32_t w_in[16])
{
    uint32_t w[16];
#pragma unroll
    for (int i = 0; i < 16; i++) w[i] = w_in[i];
    uint32_t a = st[0], b = st[1], c = st[2], d = st[3], e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll
    for (int t = 0; t < 64; t++) {
        uint32_t wt;
        if (t < 16) {
            wt = w[t];
        } else {  // the schedule kept in a ring of 16 words
            const uint32_t w15 = w[(t - 15) & 15], w2 = w[(t - 2) & 15];
            const uint32_t s0 = rotr(w15, 7) ^ rotr(w15, 18) ^ (w15 >> 3);
            const uint32_t s1 = rotr(w2, 17) ^ rotr(w2, 19) ^ (w2 >> 10);
            wt = w[t & 15] + s0 + w[(t - 7) & 15] + s1;
            w[t & 15] = wt;
        }
        const uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
        const uint32_t ch = (e & f) ^ (~e & g);
        const uint32_t T1 = h + S1 + ch + kConsts.k[t] + wt;
        const uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
        const uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
        h = g;
        g = f;
        f = e;
        e = d + T1;
        d = c;
        c = b;
        b = a;
        a = T1 + S0 + maj;
    }
    st[0] += a;
    st[1] += b;
    st[2] += c;
    st[3] += d;
    st[4] += e;
    st[5] += f;
    st[6] += g;
    st[7] += h;
}

// Byte-stream hasher (one thread).
struct Hasher {
    uint32_t st[8];
    uint8_t buf[64];
    uint32_t blen;
    uint64_t total;

    __host__ __device__ void init()
    {
        for (int i = 0; i < 8; i++) st[i] = kConsts.h[i];
        blen = 0;
        total = 0;
    }
    __host__ __device__ void block()
    {
        uint32_t w[16];
        for (int i = 0; i < 16; i++)
            w[i] = ((uint32_t)buf[4 * i] << 24) | ((uint32_t)buf[4 * i + 1] << 16) | ((uint32_t)buf[4 * i + 2] << 8) |
                   buf[4 * i + 3];
        compress(st, w);
        blen = 0;
    }
    __host__ __device__ void byte(uint8_t v)
    {
        buf[blen++] = v;
        total++;
        if (blen == 64) block();
    }
    __host__ __device__ void update(const uint8_t *p, uint64_t n)
    {
        for (uint64_t i = 0; i < n; i++) byte(p[i]);
    }
    __host__ __device__ void le(uint64_t v, int bytes)
    {
        for (int i = 0; i < bytes; i++) byte((uint8_t)(v >> (8 * i)));
    }
    // digest bytes: big-endian words
    __host__ __device__ void final(uint8_t out[32])
    {
        const uint64_t bits = total * 8;
        buf[blen++] = 0x80;
        if (blen > 56) {
            while (blen < 64) buf[blen++] = 0;
            block();
        }
        while (blen < 56) buf[blen++] = 0;
        for (int i = 0; i < 8; i++) buf[56 + i] = (uint8_t)(bits >> (56 - 8 * i));
        blen = 64;
        block();
        for (int i = 0; i < 8; i++) {
            out[4 * i] = (uint8_t)(st[i] >> 24);
            out[4 * i + 1] = (uint8_t)(st[i] >> 16);
            out[4 * i + 2] = (uint8_t)(st[i] >> 8);
            out[4 * i + 3] = (uint8_t)st[i];
        }
    }
};

__host__ __device__ inline void sha256(const uint8_t *p, uint64_t n, uint8_t out[32])
{
    Hasher h;
    h.init();
    h.update(p, n);
    h.final(out);
}

// ---- the transcript ---------------------------------------------------------
// S = H("range-arithmetic fs v1" || domain); absorb appends to the pending
// bytes Q; a draw hashes S || LE32(|Q|) || Q into S, empties Q and reads the
// challenge (LE64(S[0..8]) mod p, LE64(S[8..16]) mod p).
constexpr uint32_t kFsPending = 512;  // the most bytes pending between two draws
struct Transcript {
    uint8_t S[32];
    uint32_t qlen;
    uint8_t Q[kFsPending];
};

__host__ __device__ inline void fs_init(Transcript &t, const uint8_t domain[32])
{
    const char label[] = "range-arithmetic fs v1";
    Hasher h;
    h.init();
    h.update((const uint8_t *)label, sizeof(label) - 1);
    h.update(domain, 32);
    h.final(t.S);
    t.qlen = 0;
}

// false: more than kFsPending bytes pending
__host__ __device__ inline bool fs_absorb(Transcript &t, const uint8_t *m, uint32_t n)
{
    if (t.qlen + n > kFsPending) return false;
    for (uint32_t i = 0; i < n; i++) t.Q[t.qlen + i] = m[i];
    t.qlen += n;
    return true;
}

__host__ __device__ inline bool fs_absorb_words(Transcript &t, const uint64_t *w, uint32_t n)
{
    if (t.qlen + 8 * n > kFsPending) return false;
    for (uint32_t i = 0; i < n; i++)
        for (int b = 0; b < 8; b++) t.Q[t.qlen + 8 * i + b] = (uint8_t)(w[i] >> (8 * b));
    t.qlen += 8 * n;
    return true;
}

__host__ __device__ inline void fs_draw(Transcript &t, uint64_t out[2])
{
    Hasher h;
    h.init();
    h.update(t.S, 32);
    h.le(t.qlen, 4);
    h.update(t.Q, t.qlen);
    h.final(t.S);
    t.qlen = 0;
    constexpr uint64_t p = 0x1FFFFFFFFFFFFFFFull;
    for (int w = 0; w < 2; w++) {
        uint64_t v = 0;
        for (int i = 0; i < 8; i++) v |= (uint64_t)t.S[8 * w + i] << (8 * i);
        out[w] = v % p;
    }
}

}  // namespace sha
