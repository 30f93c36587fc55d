// fs.hip -- the non-interactive layer proof (Fiat-Shamir over F_{p^2}) on
// the device: the Merkle root of the witness tables, the transcript (absorb
// and draw, one thread: the hash chain is sequential), and the sum-check
// rounds reordered for challenges that exist only after a round's values are
// hashed.
//
// With the challenges fixed in advance (fp2.hip) a round evaluates its
// polynomial and folds its tables in the same pass.  Here the fold of round
// j - 1 has to wait for rho_{j-1}, which is the hash of round j - 1's values,
// so the pass of round j first folds (tables of 4h entries to 2h, with
// rho_{j-1}) and then evaluates round j on the folded pairs; a final fold
// after the last challenge gives the instance's final values.  A one-workgroup
// launch between the passes sums the round's partials, absorbs the values and
// draws the challenge.
#include <algorithm>

#include "common.hpp"
#include "m61.hpp"
#include "fs_device.hpp"
#include "sha256.hpp"

namespace ra {

// ---------------------------------------------------------------------------
// Merkle root: 1 KiB chunks, leaf H(0x00 || chunk), nodes H(0x01 || 4
// digests), root H(0x02 || LE64(leaves) || top).  A 4-ary node is 129 bytes
// (three compressions), which keeps the sequential levels short.
// ---------------------------------------------------------------------------
// SHA-256 of prefix || NB bytes at src (NB a multiple of 64; bytes at or
// beyond `avail` read as zero), src 16-byte aligned; digest stored as its 32
// bytes in order.
template <int NB>
__device__ void hash_chunk(uint8_t prefix, const uint8_t *__restrict__ src, uint32_t avail, uint32_t *__restrict__ out)
{
    static_assert(NB % 64 == 0, "whole blocks of data");
    uint32_t st[8];
#pragma unroll
    for (int i = 0; i < 8; i++) st[i] = sha::kConsts.h[i];
    const uint32_t *s32 = (const uint32_t *)src;
    auto word = [&](int i) -> uint32_t {  // little-endian word i of the chunk, zero past avail
        if (4u * i + 4u <= avail) return s32[i];
        uint32_t v = 0;
        for (int b = 0; b < 4; b++)
            if (4u * i + b < avail) v |= (uint32_t)src[4 * i + b] << (8 * b);
        return v;
    };
    uint32_t prev = (uint32_t)prefix << 24;  // the byte before chunk word 0 sits in the top byte
    for (int blk = 0; blk <= NB / 64; blk++) {
        uint32_t w[16];
        if (blk < NB / 64) {
            uint32_t c[16];
            if (64u * blk + 64u <= avail) {
                const uint4 *q = (const uint4 *)(src + 64 * blk);
#pragma unroll
                for (int v = 0; v < 4; v++) {
                    const uint4 x = q[v];
                    c[4 * v] = x.x;
                    c[4 * v + 1] = x.y;
                    c[4 * v + 2] = x.z;
                    c[4 * v + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int t = 0; t < 16; t++) c[t] = word(16 * blk + t);
            }
            // message word g = 16 blk + t holds bytes chunk[4g - 1], chunk[4g .. 4g + 2]
#pragma unroll
            for (int t = 0; t < 16; t++) {
                const uint32_t cw = c[t];
                w[t] = (prev & 0xFF000000u) | ((cw & 0xFFu) << 16) | (cw & 0xFF00u) | ((cw >> 16) & 0xFFu);
                prev = cw;
            }
        } else {
            // the last data byte, the 0x80 marker, zeros, the length (1 + NB) * 8 bits
            w[0] = (prev & 0xFF000000u) | 0x00800000u;
#pragma unroll
            for (int t = 1; t < 15; t++) w[t] = 0;
            w[15] = (1u + NB) * 8u;
        }
        sha::compress(st, w);
    }
#pragma unroll
    for (int i = 0; i < 8; i++) out[i] = __builtin_bswap32(st[i]);
}

__global__ __launch_bounds__(256) void k_merkle_leaves(MerkleArgs a, uint32_t *__restrict__ dig)
{
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.leaves) return;
    int sg = 0;
    while (sg < 4 && i >= a.seg[sg + 1].first_leaf) sg++;
    const uint64_t off = (i - a.seg[sg].first_leaf) * 1024;
    const uint64_t left = a.seg[sg].bytes - off;
    hash_chunk<1024>(0x00, a.seg[sg].p + off, (uint32_t)(left < 1024 ? left : 1024), dig + 8 * i);
}

__global__ __launch_bounds__(256) void k_merkle_nodes(const uint32_t *__restrict__ in, uint64_t count,
                                                      uint32_t *__restrict__ out)
{
    const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (count + 3) / 4) return;
    const uint64_t kids = std::min<uint64_t>(4, count - 4 * g);
    hash_chunk<128>(0x01, (const uint8_t *)(in + 8 * 4 * g), (uint32_t)(32 * kids), out + 8 * g);
}

__global__ void k_merkle_root(const uint32_t *__restrict__ top, uint64_t leaves, uint8_t *__restrict__ root)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    sha::Hasher h;
    h.init();
    h.byte(0x02);
    h.le(leaves, 8);
    h.update((const uint8_t *)top, 32);
    h.final(root);
}

uint64_t merkle_leaves(const MerkleArgs &a)
{
    uint64_t n = 0;
    for (int s = 0; s < 5; s++) n += (a.seg[s].bytes + 1023) / 1024;
    return n;
}

// digests: two areas of merkle_leaves() x 8 words each
void launch_merkle_root(MerkleArgs a, uint32_t *dig0, uint32_t *dig1, uint8_t *root, hipStream_t st)
{
    uint64_t first = 0;
    for (int s = 0; s < 5; s++) {
        a.seg[s].first_leaf = first;
        first += (a.seg[s].bytes + 1023) / 1024;
    }
    a.leaves = first;
    hipLaunchKernelGGL(k_merkle_leaves, dim3((unsigned)((first + 255) / 256)), dim3(256), 0, st, a, dig0);
    uint64_t count = first;
    uint32_t *in = dig0, *out = dig1;
    while (count > 1) {
        const uint64_t next = (count + 3) / 4;
        hipLaunchKernelGGL(k_merkle_nodes, dim3((unsigned)((next + 255) / 256)), dim3(256), 0, st, in, count, out);
        std::swap(in, out);
        count = next;
    }
    hipLaunchKernelGGL(k_merkle_root, dim3(1), dim3(64), 0, st, in, first, root);
}

// ---------------------------------------------------------------------------
// Transcript kernels: one thread hashes, from LDS (fs_device.hpp); a failed
// absorb sets *err.
// ---------------------------------------------------------------------------
__global__ void k_fs_header(sha::Transcript *fs, FsHeader h, const uint8_t *__restrict__ root, uint64_t *out,
                            int ndraw, uint32_t *err)
{
    __shared__ uint32_t buf32[kFsLdsBytes / 4];
    uint8_t *buf = (uint8_t *)buf32;
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    fs_pull(fs, buf);
    uint8_t r[32];
    for (int i = 0; i < 32; i++) r[i] = root[i];
    if (!fs_absorb_bytes_lds(buf, h.bytes, 64) || !fs_absorb_bytes_lds(buf, r, 32)) *err = 1;
    for (int i = 0; i < ndraw; i++) fs_draw_lds(buf, out + 2 * i);
    fs_push(fs, buf);
}

__global__ void k_fs_absorb_draw(sha::Transcript *fs, const uint64_t *__restrict__ w, int nw, uint64_t *out,
                                 int ndraw, uint32_t *err)
{
    __shared__ uint32_t buf32[kFsLdsBytes / 4];
    uint8_t *buf = (uint8_t *)buf32;
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    fs_pull(fs, buf);
    uint64_t v[16];
    for (int i = 0; i < nw && i < 16; i++) v[i] = w[i];
    if (nw > 16 || (nw && !fs_absorb_words_lds(buf, v, (uint32_t)nw))) *err = 1;
    for (int i = 0; i < ndraw; i++) fs_draw_lds(buf, out + 2 * i);
    fs_push(fs, buf);
}

// A round's values from its blocks' partials (eight words per block, the
// first nw used), written to ev; then absorbed and one challenge drawn.
__global__ __launch_bounds__(256) void k_fs_round(const uint64_t *__restrict__ part, int nb, int nw,
                                                  uint64_t *__restrict__ ev, sha::Transcript *fs, uint64_t *out,
                                                  uint32_t *err)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    __shared__ uint32_t buf32[kFsLdsBytes / 4];
    uint8_t *buf = (uint8_t *)buf32;
    if (threadIdx.x == 0) fs_pull(fs, buf);  // overlaps the sum below
    uint64_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int b = threadIdx.x; b < nb; b += blockDim.x)
#pragma unroll
        for (int q = 0; q < 8; q++) v[q] = m61::add(v[q], part[8 * (size_t)b + q]);
    m61::block_sum<8>(v, red);
    if (threadIdx.x != 0) return;
    for (int q = 0; q < nw; q++) ev[q] = v[q];
    if (!fs_absorb_words_lds(buf, v, (uint32_t)nw)) *err = 1;
    fs_draw_lds(buf, out);
    fs_push(fs, buf);
}

void launch_fs_header(sha::Transcript *fs, const FsHeader &h, const uint8_t *root, uint64_t *out, int ndraw,
                      uint32_t *err, hipStream_t st)
{
    hipLaunchKernelGGL(k_fs_header, dim3(1), dim3(64), 0, st, fs, h, root, out, ndraw, err);
}

void launch_fs_absorb_draw(sha::Transcript *fs, const uint64_t *w, int nw, uint64_t *out, int ndraw, uint32_t *err,
                           hipStream_t st)
{
    hipLaunchKernelGGL(k_fs_absorb_draw, dim3(1), dim3(64), 0, st, fs, w, nw, out, ndraw, err);
}

void launch_fs_round(const uint64_t *part, int nb, int nw, uint64_t *ev, sha::Transcript *fs, uint64_t *out,
                     uint32_t *err, hipStream_t st)
{
    hipLaunchKernelGGL(k_fs_round, dim3(1), dim3(256), 0, st, part, nb, nw, ev, fs, out, err);
}

// ---------------------------------------------------------------------------
// Rounds with the fold of the previous round first.
// ---------------------------------------------------------------------------
struct g2 {
    uint64_t re, im;
};
__device__ __forceinline__ g2 gof(uint64_t a) { return g2{a, 0}; }
__device__ __forceinline__ g2 gadd(g2 a, g2 b) { return g2{m61::add(a.re, b.re), m61::add(a.im, b.im)}; }
__device__ __forceinline__ g2 gsub(g2 a, g2 b) { return g2{m61::sub(a.re, b.re), m61::sub(a.im, b.im)}; }
__device__ __forceinline__ g2 gmul(g2 a, g2 b)
{
    const uint64_t p0 = m61::mul(a.re, b.re), p1 = m61::mul(a.im, b.im);
    const uint64_t p2 = m61::mul(m61::add(a.re, a.im), m61::add(b.re, b.im));
    return g2{m61::sub(p0, p1), m61::sub(m61::sub(p2, p0), p1)};
}
__device__ __forceinline__ g2 gld(const F2Tab &t, uint64_t i) { return g2{t.re[i], t.im[i]}; }
__device__ __forceinline__ void gst(const F2Tab &t, uint64_t i, g2 v)
{
    t.re[i] = v.re;
    t.im[i] = v.im;
}
__device__ __forceinline__ g2 gfold(g2 lo, g2 hi, g2 r) { return gadd(lo, gmul(r, gsub(hi, lo))); }

// value q of the ReLU instance read from the int32 tables: D = R - Y, S = R + Y
__device__ __forceinline__ g2 relu_int(int q, const int32_t *R, const int32_t *Y, uint64_t i)
{
    const int64_t r = R[i], y = Y[i];
    return gof(m61::from_i64(q == 1 ? r - y : r + y));
}

template <int KIND>
__global__ __launch_bounds__(256) void k_f2_round_fs(F2FsRoundArgs a)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    constexpr int NT = KIND == F2_RELU ? 3 : 2;
    g2 rho{0, 0}, ceq{0, 0}, cw{0, 0};
    if (a.fold) rho = g2{a.rho_prev[0], a.rho_prev[1]};
    if (KIND == F2_RANGE) {
        ceq = g2{a.cst[0], a.cst[1]};
        cw = g2{a.cst[2], a.cst[3]};
    }
    g2 acc[4] = {gof(0), gof(0), gof(0), gof(0)};
    const uint64_t h = a.h;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < h; i += (uint64_t)gridDim.x * blockDim.x) {
        g2 lo[3], hi[3];
#pragma unroll
        for (int q = 0; q < NT; q++) {
            const bool from_int = KIND == F2_RELU && q > 0 && a.ints;
            if (a.fold) {  // tables of 4h entries, bound at rho_{j-1}
                const g2 x0 = from_int ? relu_int(q, a.R, a.Y, i) : gld(a.src[q], i);
                const g2 x1 = from_int ? relu_int(q, a.R, a.Y, i + h) : gld(a.src[q], i + h);
                const g2 x2 = from_int ? relu_int(q, a.R, a.Y, i + 2 * h) : gld(a.src[q], i + 2 * h);
                const g2 x3 = from_int ? relu_int(q, a.R, a.Y, i + 3 * h) : gld(a.src[q], i + 3 * h);
                lo[q] = gfold(x0, x2, rho);
                hi[q] = gfold(x1, x3, rho);
                gst(a.dst[q], i, lo[q]);
                gst(a.dst[q], i + h, hi[q]);
            } else {
                lo[q] = from_int ? relu_int(q, a.R, a.Y, i) : gld(a.src[q], i);
                hi[q] = from_int ? relu_int(q, a.R, a.Y, i + h) : gld(a.src[q], i + h);
            }
        }
        g2 v[3], d[3];
#pragma unroll
        for (int q = 0; q < NT; q++) {
            v[q] = lo[q];
            d[q] = gsub(hi[q], lo[q]);
        }
#pragma unroll
        for (int X = 0; X < 4; X++) {
            if (X > 0)
#pragma unroll
                for (int q = 0; q < NT; q++) v[q] = gadd(v[q], d[q]);
            g2 f;
            if (KIND == F2_MATMUL) {
                if (X == 3) break;
                f = gmul(v[0], v[1]);
            } else if (KIND == F2_RANGE) {
                f = gmul(gmul(v[0], v[1]), gadd(gmul(ceq, gsub(v[1], gof(1))), cw));
            } else {
                f = gmul(gmul(v[0], v[1]), v[2]);
            }
            acc[X] = gadd(acc[X], f);
        }
    }
    uint64_t w[8];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        w[2 * q] = acc[q].re;
        w[2 * q + 1] = acc[q].im;
    }
    m61::block_sum<8>(w, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int q = 0; q < 8; q++) a.part[8 * (size_t)blockIdx.x + q] = w[q];
}

void launch_f2_round_fs(const F2FsRoundArgs &a, hipStream_t st)
{
    const dim3 grid(f2_blocks(a.h));
    switch (a.kind) {
    case F2_MATMUL: hipLaunchKernelGGL(k_f2_round_fs<F2_MATMUL>, grid, dim3(kThreads), 0, st, a); break;
    case F2_RANGE: hipLaunchKernelGGL(k_f2_round_fs<F2_RANGE>, grid, dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL(k_f2_round_fs<F2_RELU>, grid, dim3(kThreads), 0, st, a); break;
    }
}

// The instance's final values after its last challenge (one thread): tables
// of two entries bound at rho (or, with no rounds, their single entry).
//   F2_MATMUL  fin: c0 (g_1(0) + g_1(1), or a b with no rounds), a*, b*
//   F2_RANGE   fin: b~(sigma)
//   F2_RELU    fin: R~ = (D + S) / 2, Y~ = (S - D) / 2; ints: D, S from R, Y
__global__ void k_f2_final_fs(F2FsFinalArgs a)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    constexpr uint64_t inv2 = 1ull << 60;  // 2 2^60 = 2^61 = 1 mod p
    const int NT = a.kind == F2_RELU ? 3 : 2;
    g2 f[3];
    for (int q = 0; q < NT; q++) {
        const bool from_int = a.kind == F2_RELU && q > 0 && a.ints;
        const g2 x0 = from_int ? relu_int(q, a.R, a.Y, 0) : gld(a.t[q], 0);
        if (a.rounds > 0) {
            const g2 x1 = from_int ? relu_int(q, a.R, a.Y, 1) : gld(a.t[q], 1);
            f[q] = gfold(x0, x1, g2{a.rho[0], a.rho[1]});
        } else {
            f[q] = x0;
        }
    }
    auto put = [&](uint64_t *p, g2 v) {
        p[0] = v.re;
        p[1] = v.im;
    };
    if (a.kind == F2_MATMUL) {
        put(a.fin, a.rounds > 0 ? gadd(g2{a.ev0[0], a.ev0[1]}, g2{a.ev0[2], a.ev0[3]}) : gmul(f[0], f[1]));
        put(a.fin + 2, f[0]);
        put(a.fin + 4, f[1]);
    } else if (a.kind == F2_RANGE) {
        put(a.fin, f[1]);
    } else {
        const g2 D = f[1], S = f[2];
        put(a.fin, g2{m61::mul(m61::add(D.re, S.re), inv2), m61::mul(m61::add(D.im, S.im), inv2)});
        put(a.fin + 2, g2{m61::mul(m61::sub(S.re, D.re), inv2), m61::mul(m61::sub(S.im, D.im), inv2)});
    }
}

void launch_f2_final_fs(const F2FsFinalArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_final_fs, dim3(1), dim3(64), 0, st, a);
}

// Bx(x) = sum over the set bits q of word x of eq(sigma_p, q): the bit table
// bound at the plane challenges (both parts), eq(sigma_p, .) staged in LDS.
__global__ __launch_bounds__(256) void k_f2_bx(const uint64_t *__restrict__ bits, uint64_t N, F2Tab SIG, int P,
                                               F2Tab Bx)
{
    __shared__ uint64_t sre[64], sim[64];
    if (threadIdx.x < 64) {
        sre[threadIdx.x] = (int)threadIdx.x < P ? SIG.re[threadIdx.x] : 0;
        sim[threadIdx.x] = (int)threadIdx.x < P ? SIG.im[threadIdx.x] : 0;
    }
    __syncthreads();
    for (uint64_t x = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < N; x += (uint64_t)gridDim.x * blockDim.x) {
        uint64_t w = bits[x], re = 0, im = 0;
        while (w) {
            const int q = __builtin_ctzll(w);
            w &= w - 1;
            re = m61::add(re, sre[q]);
            im = m61::add(im, sim[q]);
        }
        Bx.re[x] = re;
        Bx.im[x] = im;
    }
}

void launch_f2_bx(const uint64_t *bits, uint64_t N, F2Tab SIG, int P, F2Tab Bx, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_bx, dim3(f2_blocks(N)), dim3(kThreads), 0, st, bits, N, SIG, P, Bx);
}

__global__ __launch_bounds__(256) void k_fill0(uint64_t *__restrict__ p, uint64_t n)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

void launch_fill0(uint64_t *p, uint64_t n, hipStream_t st)
{
    hipLaunchKernelGGL(k_fill0, dim3(f2_blocks(n)), dim3(kThreads), 0, st, p, n);
}

}  // namespace ra
