// fs_device.hpp -- the Fiat-Shamir transcript on the device, worked by one
// thread from LDS.  The transcript (sha::Transcript in device memory: S,
// the pending length, the pending bytes) is pulled into an LDS buffer laid
// out as the next draw's message, S || LE32(|Q|) || Q, so that absorbing
// appends to it and drawing hashes it in place; it is pushed back once at the
// end of the kernel.  (Byte-wise work on device memory would put a memory
// round trip on every byte of the sequential hash chain.)
#pragma once
#include "sha256.hpp"

namespace ra {

constexpr uint32_t kFsLdsBytes = 36 + sha::kFsPending + 64;  // the message, with room for the padding

// SHA-256 of the len bytes at m (LDS, 4-byte aligned) into st.
__device__ inline void sha256_lds(const uint8_t *m, uint32_t len, uint32_t st[8])
{
    for (int i = 0; i < 8; i++) st[i] = sha::kConsts.h[i];
    const uint32_t nblk = (len + 9 + 63) / 64;
    const uint64_t bits = (uint64_t)len * 8;
    const uint32_t *m32 = (const uint32_t *)m;
    for (uint32_t b = 0; b < nblk; b++) {
        uint32_t w[16];
        for (int t = 0; t < 16; t++) {
            const uint32_t j = 64 * b + 4 * t;
            if (j + 4 <= len) {
                w[t] = __builtin_bswap32(m32[j / 4]);
            } else if (b == nblk - 1 && t >= 14) {
                w[t] = t == 14 ? (uint32_t)(bits >> 32) : (uint32_t)bits;
            } else {
                uint32_t v = 0;
                for (int u = 0; u < 4; u++) {
                    const uint32_t q = j + u;
                    v = (v << 8) | (q < len ? m[q] : (q == len ? 0x80u : 0u));
                }
                w[t] = v;
            }
        }
        sha::compress(st, w);
    }
}

// One thread: the transcript into buf (S, LE32 qlen, Q).
__device__ inline void fs_pull(const sha::Transcript *g, uint8_t *buf)
{
    const uint32_t *s = (const uint32_t *)g;
    uint32_t *d = (uint32_t *)buf;
    const uint32_t qlen = g->qlen;
    const uint32_t words = (36 + qlen + 3) / 4;
    for (uint32_t i = 0; i < words; i++) d[i] = s[i];
}

__device__ inline uint32_t fs_qlen(const uint8_t *buf) { return *(const uint32_t *)(buf + 32); }

// false: more than sha::kFsPending bytes pending
__device__ inline bool fs_absorb_words_lds(uint8_t *buf, const uint64_t *w, uint32_t n)
{
    uint32_t q = fs_qlen(buf);
    if (q + 8 * n > sha::kFsPending) return false;
    for (uint32_t i = 0; i < n; i++)
        for (int b = 0; b < 8; b++) buf[36 + q + 8 * i + b] = (uint8_t)(w[i] >> (8 * b));
    *(uint32_t *)(buf + 32) = q + 8 * n;
    return true;
}

__device__ inline bool fs_absorb_bytes_lds(uint8_t *buf, const uint8_t *m, uint32_t n)
{
    uint32_t q = fs_qlen(buf);
    if (q + n > sha::kFsPending) return false;
    for (uint32_t i = 0; i < n; i++) buf[36 + q + i] = m[i];
    *(uint32_t *)(buf + 32) = q + n;
    return true;
}

// A draw: S = H(S || LE32(|Q|) || Q), Q emptied, the challenge's two words.
__device__ inline void fs_draw_lds(uint8_t *buf, uint64_t out[2])
{
    uint32_t st[8];
    sha256_lds(buf, 36 + fs_qlen(buf), st);
    uint32_t *s32 = (uint32_t *)buf;
    for (int i = 0; i < 8; i++) s32[i] = __builtin_bswap32(st[i]);  // S as its bytes in order
    s32[8] = 0;
    constexpr uint64_t p = 0x1FFFFFFFFFFFFFFFull;
    for (int w = 0; w < 2; w++) {
        const uint64_t v = (uint64_t)s32[2 * w] | ((uint64_t)s32[2 * w + 1] << 32);  // LE64 of S[8w .. 8w + 8]
        const uint64_t r = (v & p) + (v >> 61);                                       // v mod p (v < 2^64)
        out[w] = r >= p ? r - p : r;
    }
}

// One thread: buf back into the transcript.
__device__ inline void fs_push(sha::Transcript *g, const uint8_t *buf)
{
    const uint32_t *s = (const uint32_t *)buf;
    uint32_t *d = (uint32_t *)g;
    const uint32_t words = (36 + fs_qlen(buf) + 3) / 4;
    for (uint32_t i = 0; i < words; i++) d[i] = s[i];
}

}  // namespace ra
