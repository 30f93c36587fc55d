// planes.hip -- the plane rounds of the concatenated range check.
//
// Over the bit table b(q, x) (q = plane, the first log P variables; x the
// output index) the range summand is
//   eq(tau_p, q) EQ(x) b (b - 1) + mu W(q) EQ(x) b,     EQ(x) = eq((r1, r2), x).
// While plane variable j is free and x is still Boolean, the round
// polynomial is g_j(X) = K_j eq(tau_j, X) A_j(X) + mu Bw_j(X) with
//   A_j(X)  = sum_p' e_j[p'] sum_x EQ(x) (b_X^2 - b_X),
//   Bw_j(X) = sum_p' W_j(X, p') sum_x EQ(x) b_X,
// b_X = b(sigma_<j, X, p', x) = sum_y c_y bit_(y, X, p')(x), c_y = eq(sigma_<j, y).
// Every x-sum above is a linear combination of the entries of the Gram
// matrix G[q][q'] = sum_x EQ(x) bit_q(x) bit_q'(x) (its diagonal gives the
// linear terms, since a bit squared is itself).  G is an exact integer
// contraction over x, so it runs on the matrix cores: EQ(x) is written in
// eight balanced base-256 digits d_t(x) in [-128, 128), and
// G_t = Bits^T diag(d_t) Bits is an int8 x int8 -> int32 product
// (v_mfma_i32_16x16x64_i8 over the 16 x 16 tiles on and above the diagonal:
// G is symmetric), recombined as sum_t 256^t G_t modulo p.  The
// same pass writes the plane-bound table Bx(x) = sum_q eq(sigma_p, q) bit_q(x)
// (eight byte lookups per x), the input of the rounds over x.
#include "common.hpp"
#include "m61.hpp"
#include "gram_reduce.hpp"
#include "rsetup.hpp"

namespace ra {

typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int kLimbs = 8;    // balanced base-256 digits of a field element


// Block layout of the Gram pass: sixteen waves with two roles, working on
// slabs of kSlab outputs through a double-buffered LDS area.
//   producers (waves 0-7, one output per thread): EQ(x), Bx and the digits
//     of EQ(x); the bit words turned plane-major: in each group of eight
//     lanes (outputs) every byte's 8 x 8 bit block is transposed across the
//     lanes, so a lane holds one plane's bits for eight outputs per byte,
//     stored as bytes 0x00 / 0xFF in rows padded so that the matrix-core
//     fragment reads are free of bank conflicts;
//   consumers (waves 8-15, two per SIMD): wave c accumulates digit c for
//     every 16 x 16 tile of G on or above the diagonal over the slab's
//     K-steps of 64 outputs on the matrix cores.
// While the consumers stream slab i the producers build slab i + 1; one
// barrier per slab hands the buffers over.  While the producers build the
// first slab the consumers are free: with xs_on they run the set-up of the
// range call's rounds over x (xsetup.hpp), one entry per consumer thread.
constexpr int kSlab = 512;
constexpr int kRow = kSlab + 16;  // bytes per plane row in LDS
constexpr int kProducers = 8, kConsumers = 8, kGramThreads = 64 * (kProducers + kConsumers);

// NPL planes (32 or 64) in NB = NPL / 16 blocks of sixteen; tile t < NT
// covers plane blocks (I, J), I <= J, in the order (0,0), (0,1), .., (1,1), ..
template <int NPL> struct GramShape {
    static constexpr int kBlocks = NPL / 16;
    static constexpr int kTiles = kBlocks * (kBlocks + 1) / 2;
    static_assert(kLimbs == kConsumers, "one digit per consumer wave");
};

// 8 x 8 bit transposes across each group of eight lanes, one per byte of a
// 32-bit word: lane 8 g + i holds row i of every byte's block (bit k of byte
// b = entry (i, k)) and ends with column i (bit k of byte b = entry (k, i)).
// Three butterfly stages, each swapping the off-diagonal j x j blocks of
// every 2j x 2j block with the partner lane i ^ j, taken by DPP moves:
// xor 1 and xor 2 are quad permutations, xor 4 a half-row mirror followed by
// a quad reversal (lane i -> 7 - i -> 7 - (i ^ 3) = i ^ 4).
__device__ __forceinline__ uint32_t dpp_xor1(uint32_t v) { return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false); }
__device__ __forceinline__ uint32_t dpp_xor2(uint32_t v) { return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false); }
__device__ __forceinline__ uint32_t dpp_xor4(uint32_t v)
{
    return __builtin_amdgcn_mov_dpp(__builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false), 0x1B, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t butterfly(uint32_t a, uint32_t b, bool upper, int j, uint32_t m)
{
    return upper ? ((a & ~m) | ((b & ~m) >> j)) : ((a & m) | ((b & m) << j));
}
__device__ __forceinline__ uint32_t byte_blocks_transpose(uint32_t a)
{
    const int lane = threadIdx.x & 63;
    a = butterfly(a, dpp_xor4(a), lane & 4, 4, 0x0F0F0F0Fu);
    a = butterfly(a, dpp_xor2(a), lane & 2, 2, 0x33333333u);
    return butterfly(a, dpp_xor1(a), lane & 1, 1, 0x55555555u);
}

// Balanced base-256 digits of e < 2^62: e = sum_t 256^t d_t, d_t in [-128, 128).
// With f = e + sum_t 128 256^t (no overflow: e < 2^62), the plain bytes f_t
// give d_t = f_t - 128, whose int8 bit pattern is f_t with the top bit flipped;
// so the eight digit bytes are those of f xor 0x80...80.  The digits add up to
// e itself, so a folded (not canonical) e gives the same G modulo p.
__device__ __forceinline__ uint64_t balanced_digit_bytes(uint64_t e)
{
    constexpr uint64_t kHalf = 0x8080808080808080ull;
    return (e + kHalf) ^ kHalf;
}

template <int NPL>
__global__ __launch_bounds__(kGramThreads) void k_plane_gram(
    const uint64_t *__restrict__ bits, uint64_t N, int lk, const uint64_t *__restrict__ E1,
    const uint64_t *__restrict__ E2, const uint64_t *__restrict__ sig, int lP, uint64_t *__restrict__ Bx,
    uint64_t *__restrict__ gpart, int xs_on, XSetupArgs xs, const uint64_t *__restrict__ eqs)
{
    using S = GramShape<NPL>;
    constexpr int NB = S::kBlocks, NT = S::kTiles;
    constexpr int kPlaneBytes = NPL * kRow, kTileBytes = NT * kGramTileWords * 8;
    static_assert(2 * kPlaneBytes >= kTileBytes, "the tiles reuse the plane buffers");
    __shared__ uint64_t s_lut[8 * 256];                                    // Bx byte tables
    __shared__ uint64_t s_eqs[64];                                         // eq(sigma_p, q)
    __shared__ uint64_t s_exp[256];                                        // byte -> eight 0x00 / 0xFF bytes
    __shared__ __attribute__((aligned(16))) int8_t s_d[2][kLimbs][kSlab];  // digits of EQ(x)
    // plane bytes of two slabs; afterwards the block's Gram tiles (tile t,
    // entry 64 r + lane of fragment register r)
    __shared__ __attribute__((aligned(16))) int8_t s_u[2 * kPlaneBytes];
    unsigned long long(*s_g)[kGramTileWords] = (unsigned long long(*)[kGramTileWords])s_u;
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool producer = wv < kProducers;  // wave-uniform
    const int cw = wv - kProducers;         // consumer index = its digit
    if (tid < 64) {  // eq(sigma_p, q) for every plane q (or the given values)
        uint64_t a = 0;
        if (tid < (1 << lP)) {
            if (eqs) {
                a = eqs[tid];
            } else {  // the point's coordinates loaded together, then the products
                uint64_t zs[kMaxPlaneLog];
#pragma unroll
                for (int i = 0; i < kMaxPlaneLog; i++) zs[i] = i < lP ? sig[i] : 0;
                a = 1;
#pragma unroll
                for (int i = 0; i < kMaxPlaneLog; i++)
                    if (i < lP) a = m61::lmul(a, ((tid >> (lP - 1 - i)) & 1) ? zs[i] : m61::lsub(1, zs[i]));
            }
        }
        s_eqs[tid] = m61::canon(a);
    }
    for (int i = tid; i < 256; i += kGramThreads) {
        uint64_t e = 0;
        for (int b = 0; b < 8; b++)
            if ((i >> b) & 1) e |= 0xFFull << (8 * b);
        s_exp[i] = e;
    }
    const uint64_t kmask = (1ull << lk) - 1;
    const uint64_t nslabs = (N + kSlab - 1) / kSlab;
    const uint64_t mine = nslabs > blockIdx.x ? (nslabs - blockIdx.x + gridDim.x - 1) / gridDim.x : 0;
    // a slab's global inputs are read one slab ahead; the first slab's before
    // the byte tables are built
    uint64_t pw = 0, pe1 = 0, pe2 = 0;
    auto fetch = [&](uint64_t i) {
        const uint64_t x = (blockIdx.x + i * gridDim.x) * kSlab + tid;
        const bool valid = i < mine && x < N;
        pw = valid ? bits[x] : 0;
        pe1 = valid ? E1[x >> lk] : 0;
        pe2 = valid ? E2[x & kmask] : 0;
    };
    if (producer) fetch(0);
    // With xs_on the consumer waves also run the set-up of the rounds over x
    // (it depends on challenges only) while the producers build the first
    // slab; its challenges are staged here.
    __shared__ uint64_t s_xr[64], s_xs[64], s_xz[64];
    if (xs_on && tid < xs.lN) {
        s_xr[tid] = xs.r[tid];
        s_xs[tid] = xs.sigx[tid];
        s_xz[tid] = xs.rho2 ? xs.rho2[tid] : 0;
    }
    __syncthreads();
    // byte tables of Bx(x) = sum_q eq(sigma_p, q) bit_q(x): lut[b][v] = sum
    // over the set bits i of v of eq(sigma_p, 8 b + i)
    for (int i = tid; i < 8 * 256; i += kGramThreads) {
        const int b = i >> 8, v = i & 255;
        uint64_t a = 0;
        for (int k = 0; k < 8; k++)
            if ((v >> k) & 1) a += s_eqs[8 * b + k];  // eight values below 2^61
        s_lut[i] = m61::canon(a);
    }
    __syncthreads();  // byte tables ready
    // The two roles run separate loops with the same barriers (one per slab),
    // so the consumers' accumulators are not live in the producers' code.
    if (producer) {
        for (uint64_t i = 0; i <= mine; i++) {
            if (i < mine) {  // build slab i into buffer i % 2
                const int buf = (int)(i & 1);
                const uint64_t x = (blockIdx.x + i * gridDim.x) * kSlab + tid;
                const bool valid = x < N;
                const uint64_t w = pw, eqx = m61::lmul(pe1, pe2);  // folded, < 2^61 + 8
                fetch(i + 1);
                uint64_t bx = 0;  // eight values below 2^61: the plain sum stays below 2^64
#pragma unroll
                for (int b = 0; b < 8; b++) bx += s_lut[b * 256 + ((w >> (8 * b)) & 255)];
                if (valid) Bx[x] = m61::reduce64(bx);
                const uint64_t db = balanced_digit_bytes(eqx);
#pragma unroll
                for (int t = 0; t < kLimbs; t++) s_d[buf][t][tid] = (int8_t)(db >> (8 * t));
                // lane 8 g + i: byte b = plane 8 b + i over outputs 8 g .. 8 g + 7
                // of the wave, stored as eight 0x00 / 0xFF bytes in that plane's row
                const uint32_t lo = byte_blocks_transpose((uint32_t)w), hi = byte_blocks_transpose((uint32_t)(w >> 32));
                int8_t *col = s_u + buf * kPlaneBytes + (lane & 7) * kRow + (tid & ~63) + 8 * (lane >> 3);
#pragma unroll
                for (int b = 0; b < NPL / 8; b++)
                    *(uint64_t *)(col + 8 * b * kRow) = s_exp[((b < 4 ? lo : hi) >> (8 * (b & 3))) & 255];
            }
            __syncthreads();
        }
        __syncthreads();  // the consumers have cleared the tiles
        __syncthreads();  // and added their digits
    } else {
        // whole waves of the set-up, spread one wave per block before a block's
        // second wave (wave w of block b takes entries 64 (w B + b) ..)
        if (xs_on) x_setup_body(xs, (int)(((wv - kProducers) * gridDim.x + blockIdx.x) * 64) + lane, s_xr, s_xs, s_xz);
        v4i acc[NT];
#pragma unroll
        for (int t = 0; t < NT; t++) acc[t] = v4i{0, 0, 0, 0};
        for (uint64_t i = 0; i <= mine; i++) {
            if (i > 0) {  // consume slab i - 1 from buffer (i - 1) % 2
                const int buf = (int)((i - 1) & 1);
                // K-step ks covers outputs 64 ks .. 64 ks + 63 of the slab; lane l
                // holds row l % 16 of a 16-row block and the sixteen outputs
                // 16 (l / 16) .. of the step, as do the digit bytes it reads
                const int8_t *frow = s_u + buf * kPlaneBytes + (lane & 15) * kRow + 16 * (lane >> 4);
                const int8_t *drow = &s_d[buf][cw][16 * (lane >> 4)];
                // The plane bytes are 0x00 / 0xFF, i.e. -bit as int8: they are the
                // A operand as they stand (the tiles accumulate -G_t, negated in
                // the recombination), and masked with the digits they give B.
                // Two register sets alternate over the K-steps, so the reads of
                // step ks + 1 are in flight during the products of step ks.
                v4i f0[NB], d0, f1[NB], d1;
                auto load = [&](v4i (&f)[NB], v4i &d, int ks) {
#pragma unroll
                    for (int I = 0; I < NB; I++) f[I] = *(const v4i *)(frow + 16 * I * kRow + 64 * ks);
                    d = *(const v4i *)(drow + 64 * ks);
                };
                auto step = [&](const v4i (&f)[NB], const v4i &d) {
                    v4i bj[NB];
#pragma unroll
                    for (int J = 0; J < NB; J++) bj[J] = f[J] & d;
                    int t = 0;
#pragma unroll
                    for (int I = 0; I < NB; I++)
#pragma unroll
                        for (int J = I; J < NB; J++, t++)
                            acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(f[I], bj[J], acc[t], 0, 0, 0);
                };
                static_assert((kSlab / 64) % 2 == 0, "K-steps come in pairs");
                load(f0, d0, 0);
                for (int ks = 0; ks < kSlab / 64; ks += 2) {
                    load(f1, d1, ks + 1);
                    step(f0, d0);
                    if (ks + 2 < kSlab / 64) load(f0, d0, ks + 2);
                    step(f1, d1);
                }
            }
            __syncthreads();
        }
        // recombine the digits modulo p into the block's tiles: digit t weighs
        // 2^(8t), a rotation of the 61-bit residue (of -acc: the A operand
        // held -bit); one LDS atomic per entry
        // and consumer wave (8 waves x values below 2^61 < 2^64)
        for (int i = tid - 64 * kProducers; i < NT * kGramTileWords; i += 64 * kConsumers) (&s_g[0][0])[i] = 0;
        __syncthreads();
#pragma unroll
        for (int t = 0; t < NT; t++)
#pragma unroll
            for (int r = 0; r < 4; r++)
                atomicAdd(&s_g[t][r * 64 + lane], (unsigned long long)m61::rotl(m61::from_i32(-acc[t][r]), 8 * cw));
        __syncthreads();
    }
    for (int i = tid; i < NT * kGramTileWords; i += kGramThreads)
        gpart[(size_t)blockIdx.x * NT * kGramTileWords + i] = m61::reduce64((&s_g[0][0])[i]);
}

// Sum of the blocks' partial tiles, written as G[q][q'] (64 x 64, both
// triangles).  Each block covers 64 tile entries; its four waves split the
// partial blocks and combine through LDS.
// The range call's set-up as a launch of its own, for tables too small for a
// register pass (otherwise these roles ride elsewhere: the set-up of the
// rounds over x in the Gram pass, the rest in the first register pass).
// Workgroups below nred: 16 entries of G each (gram_reduce.hpp).  The next
// workgroup writes the constant block of the plane rounds, with a deferred
// witness step the one after sums the witness claims (and the claimed sum of
// the range instance), the others run the set-up of the rounds over x.
__global__ __launch_bounds__(256) void k_gram_reduce(const uint64_t *__restrict__ gpart, int nblk, int tiles,
                                                     uint64_t *__restrict__ G, int nred, RangeConsts rc,
                                                     XSetupArgs xs)
{
    const int ncj = rc.cj.nblk > 0 ? 1 : 0;  // a deferred witness step: one more workgroup
    if ((int)blockIdx.x > nred + ncj) {
        x_setup_block(xs, blockIdx.x - nred - 1 - ncj);
        return;
    }
    if (ncj && (int)blockIdx.x == nred + 1) {
        witness_claims_block(rc);
        return;
    }
    if ((int)blockIdx.x == nred) {
        range_consts_block(rc);
        return;
    }
    __shared__ uint64_t red[kGramReduceLdsWords];
    gram_reduce_block(gpart, nblk, tiles, G, blockIdx.x, red);
}

int plane_gram_tiles(int lP, int pused)
{
    if (lP <= 5) return GramShape<32>::kTiles;
    return pused <= 48 ? GramShape<48>::kTiles : GramShape<64>::kTiles;
}

int plane_gram_set_up_threads(uint64_t N, int lP) { return plane_gram_blocks(N, lP) * 64 * kConsumers; }

int plane_gram_blocks(uint64_t N, int lP)
{
    (void)lP;
    const uint64_t slabs = (N + kSlab - 1) / kSlab;
    return (int)(slabs < 256 ? slabs : 256);
}

void launch_plane_gram(int lP, const uint64_t *bits, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2,
                       const uint64_t *sig, uint64_t *Bx, uint64_t *gpart, const XSetupArgs *xs, hipStream_t st,
                       const uint64_t *eqs, int pused)
{
    const int nb = plane_gram_blocks(N, lP);
    const XSetupArgs none{};
    const XSetupArgs &x = xs ? *xs : none;
    if (lP <= 5)
        hipLaunchKernelGGL(k_plane_gram<32>, dim3(nb), dim3(kGramThreads), 0, st, bits, N, lk, E1, E2, sig, lP, Bx,
                           gpart, xs ? 1 : 0, x, eqs);
    else if (plane_gram_tiles(lP, pused) == GramShape<48>::kTiles)  // planes 48 .. 63 are zero
        hipLaunchKernelGGL(k_plane_gram<48>, dim3(nb), dim3(kGramThreads), 0, st, bits, N, lk, E1, E2, sig, lP, Bx,
                           gpart, xs ? 1 : 0, x, eqs);
    else
        hipLaunchKernelGGL(k_plane_gram<64>, dim3(nb), dim3(kGramThreads), 0, st, bits, N, lk, E1, E2, sig, lP, Bx,
                           gpart, xs ? 1 : 0, x, eqs);
}

void launch_gram_reduce(int lP, uint64_t N, const uint64_t *gpart, uint64_t *gsum, const RangeConsts &rc,
                        const XSetupArgs &xs, hipStream_t st, int pused)
{
    const int tiles = plane_gram_tiles(lP, pused), nb = plane_gram_blocks(N, lP), nred = gram_reduce_groups(tiles);
    const int xb = (x_setup_count(xs) + 255) / 256;
    const int ncj = rc.cj.nblk > 0 ? 1 : 0;
    hipLaunchKernelGGL(k_gram_reduce, dim3(nred + 1 + ncj + xb), dim3(256), 0, st, gpart, nb, tiles, gsum, nred, rc,
                       xs);
}

}  // namespace ra
