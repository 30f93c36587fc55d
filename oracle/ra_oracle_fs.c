/*
 * ra_oracle_fs.c -- the Fiat-Shamir transcript that makes the layer protocol
 * non-interactive: the verifier's challenges are hashes of everything the
 * prover has sent before them.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; it shares no code with the GPU path.
 *
 * The paper's protocol is interactive (the verifier picks the sum-check
 * challenges, Sec. II-D; Alg. 1).  The transform used here, one of the
 * standard readings, is:
 *
 *   hash H = SHA-256 (FIPS 180-4);
 *   S_0 = H("range-arithmetic fs v1" || domain), domain 32 caller bytes;
 *   absorb(M): append M to the pending bytes Q;
 *   draw():    S = H(S || LE32(|Q|) || Q), Q = empty, and the challenge is
 *              (LE64(S[0..8]) mod p) + (LE64(S[8..16]) mod p) i in F_{p^2};
 *   F_{p^2} elements are absorbed as LE64(re) || LE64(im), integers as LE32.
 *
 * The witness tables, which the prover picks, are bound before any challenge
 * that depends on them: their Merkle root is absorbed with the layer header.
 * Root over the tables R (LE32), Rm (LE16), Y (LE32), Z (LE32) and the packed
 * bit table (N LE64 words, bit q of word x = plane q), each zero-padded to a
 * multiple of 1024 bytes and concatenated: chunk i of 1024 bytes gives the
 * leaf H(0x00 || chunk_i); while more than one digest remains, consecutive
 * digests are grouped by 4 (the last group zero-filled) into H(0x01 || 4
 * digests); the root is H(0x02 || LE64(leaves) || top).
 *
 * SHA-256 follows FIPS 180-4 Sec. 4-6; its constants are computed from their
 * definition (the first 32 bits of the fractional parts of the square roots
 * of the first 8 primes, and of the cube roots of the first 64 primes).
 */
#include "ra_oracle_fs.h"

#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define FS_P ((uint64_t)0x1FFFFFFFFFFFFFFFULL)

/* ------------------------------------------------------------------------ */
/* SHA-256                                                                   */
/* ------------------------------------------------------------------------ */
static uint32_t H0[8], K[64];
static int consts_ready;

static u128 iroot(u128 v, int e)
{
    /* the largest x with x^e <= v (e = 2 or 3), by bisection */
    u128 lo = 0, hi = (u128)1 << (e == 2 ? 64 : 43);
    while (lo < hi) {
        u128 mid = lo + (hi - lo + 1) / 2, p = mid * mid;
        if (e == 3) p *= mid;
        if (p <= v) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

static void make_constants(void)
{
    int primes[64], n = 0;
    for (int x = 2; n < 64; x++) {
        int prime = 1;
        for (int d = 2; d * d <= x; d++)
            if (x % d == 0) prime = 0;
        if (prime) primes[n++] = x;
    }
    for (int i = 0; i < 8; i++) H0[i] = (uint32_t)iroot((u128)primes[i] << 64, 2);
    for (int i = 0; i < 64; i++) K[i] = (uint32_t)iroot((u128)primes[i] << 96, 3);
    consts_ready = 1;
}

static uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

static void compress(uint32_t h[8], const uint8_t block[64])
{
    uint32_t W[64];
    for (int t = 0; t < 16; t++)
        W[t] = ((uint32_t)block[4 * t] << 24) | ((uint32_t)block[4 * t + 1] << 16) |
               ((uint32_t)block[4 * t + 2] << 8) | block[4 * t + 3];
    for (int t = 16; t < 64; t++) {
        uint32_t s0 = rotr(W[t - 15], 7) ^ rotr(W[t - 15], 18) ^ (W[t - 15] >> 3);
        uint32_t s1 = rotr(W[t - 2], 17) ^ rotr(W[t - 2], 19) ^ (W[t - 2] >> 10);
        W[t] = s1 + W[t - 7] + s0 + W[t - 16];
    }
    uint32_t a = h[0], b = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], hh = h[7];
    for (int t = 0; t < 64; t++) {
        uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
        uint32_t ch = (e & f) ^ (~e & g);
        uint32_t T1 = hh + S1 + ch + K[t] + W[t];
        uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
        uint32_t maj = (a & b) ^ (a & c) ^ (b & c);
        uint32_t T2 = S0 + maj;
        hh = g;
        g = f;
        f = e;
        e = d + T1;
        d = c;
        c = b;
        b = a;
        a = T1 + T2;
    }
    h[0] += a;
    h[1] += b;
    h[2] += c;
    h[3] += d;
    h[4] += e;
    h[5] += f;
    h[6] += g;
    h[7] += hh;
}

void orc_sha256(const uint8_t *msg, size_t len, uint8_t out[32])
{
    if (!consts_ready) make_constants();
    uint32_t h[8];
    memcpy(h, H0, sizeof(h));
    size_t full = len / 64;
    for (size_t i = 0; i < full; i++) compress(h, msg + 64 * i);
    /* padding: 0x80, zeros, the bit length as a 64-bit big-endian integer */
    uint8_t tail[128];
    size_t rem = len - 64 * full;
    memset(tail, 0, sizeof(tail));
    memcpy(tail, msg + 64 * full, rem);
    tail[rem] = 0x80;
    size_t tl = rem + 1 + 8 <= 64 ? 64 : 128;
    uint64_t bits = (uint64_t)len * 8;
    for (int i = 0; i < 8; i++) tail[tl - 1 - i] = (uint8_t)(bits >> (8 * i));
    compress(h, tail);
    if (tl == 128) compress(h, tail + 64);
    for (int i = 0; i < 8; i++) {
        out[4 * i] = (uint8_t)(h[i] >> 24);
        out[4 * i + 1] = (uint8_t)(h[i] >> 16);
        out[4 * i + 2] = (uint8_t)(h[i] >> 8);
        out[4 * i + 3] = (uint8_t)h[i];
    }
}

/* ------------------------------------------------------------------------ */
/* Transcript                                                                */
/* ------------------------------------------------------------------------ */
void orc_fs_init(orc_fs *t, const uint8_t domain[32])
{
    static const char label[] = "range-arithmetic fs v1";
    uint8_t buf[64];
    size_t ll = strlen(label);
    memcpy(buf, label, ll);
    memcpy(buf + ll, domain, 32);
    orc_sha256(buf, ll + 32, t->S);
    t->qlen = 0;
}

int orc_fs_absorb(orc_fs *t, const uint8_t *m, uint32_t len)
{
    if (t->qlen + len > sizeof(t->Q)) return -1;
    memcpy(t->Q + t->qlen, m, len);
    t->qlen += len;
    return 0;
}

void orc_fs_draw(orc_fs *t, uint64_t out[2])
{
    uint8_t buf[32 + 4 + sizeof(t->Q)];
    memcpy(buf, t->S, 32);
    for (int i = 0; i < 4; i++) buf[32 + i] = (uint8_t)(t->qlen >> (8 * i));
    memcpy(buf + 36, t->Q, t->qlen);
    orc_sha256(buf, 36 + (size_t)t->qlen, t->S);
    t->qlen = 0;
    for (int w = 0; w < 2; w++) {
        uint64_t v = 0;
        for (int i = 0; i < 8; i++) v |= (uint64_t)t->S[8 * w + i] << (8 * i);
        out[w] = v % FS_P;
    }
}

/* ------------------------------------------------------------------------ */
/* Merkle root of the witness tables                                         */
/* ------------------------------------------------------------------------ */
static void put_le(uint8_t *p, uint64_t v, int bytes)
{
    for (int i = 0; i < bytes; i++) p[i] = (uint8_t)(v >> (8 * i));
}

int orc_witness_root(const int64_t *R, const int64_t *Rm, const int64_t *Y, const int64_t *Z, const uint64_t *words,
                     int64_t N, uint8_t out[32])
{
    const int64_t *tabs[4] = {R, Rm, Y, Z};
    const int width[5] = {4, 2, 4, 4, 8};
    size_t padded[5], total = 0;
    for (int i = 0; i < 5; i++) {
        size_t b = (size_t)N * width[i];
        padded[i] = (b + 1023) / 1024 * 1024;
        total += padded[i];
    }
    uint8_t *data = calloc(total > 0 ? total : 1, 1);
    if (!data) return -10;
    size_t off = 0;
    for (int i = 0; i < 5; i++) {
        for (int64_t x = 0; x < N; x++)
            put_le(data + off + (size_t)x * width[i], i < 4 ? (uint64_t)tabs[i][x] : words[x], width[i]);
        off += padded[i];
    }
    size_t count = total / 1024;
    uint8_t *dig = malloc(32 * (count > 0 ? count : 1)), buf[1 + 1024];
    if (!dig) {
        free(data);
        return -10;
    }
    for (size_t i = 0; i < count; i++) {
        buf[0] = 0x00;
        memcpy(buf + 1, data + 1024 * i, 1024);
        orc_sha256(buf, sizeof(buf), dig + 32 * i);
    }
    size_t leaves = count;
    while (count > 1) {
        size_t next = (count + 3) / 4;
        for (size_t g = 0; g < next; g++) {
            uint8_t node[1 + 4 * 32];
            memset(node, 0, sizeof(node));
            node[0] = 0x01;
            for (size_t c = 0; c < 4 && 4 * g + c < count; c++) memcpy(node + 1 + 32 * c, dig + 32 * (4 * g + c), 32);
            orc_sha256(node, sizeof(node), dig + 32 * g); /* g <= 4 g: the group's inputs are already read */
        }
        count = next;
    }
    uint8_t fin[1 + 8 + 32];
    fin[0] = 0x02;
    put_le(fin + 1, (uint64_t)leaves, 8);
    memcpy(fin + 9, dig, 32);
    orc_sha256(fin, sizeof(fin), out);
    free(dig);
    free(data);
    return 0;
}
