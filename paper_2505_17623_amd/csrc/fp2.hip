// fp2.hip -- the layer protocol with the verifier's challenges in the
// quadratic extension F_{p^2} = F_p[i] / (i^2 + 1) (p = 2^61 - 1 is 3 mod 4,
// so x^2 + 1 is irreducible).  Sec. II-F asks for a field of more than 128
// bits; a sum-check round over F_{p^2} lets a cheating prover pass with
// probability about d / p^2 instead of d / p (Sec. II-D).
//
// The witness (C, R, Rm, Y, Z, the bit table) is integer-valued and is made
// by the F_p kernels.  Everything that depends on a challenge is an element
// of F_{p^2}, held as two F_p tables (real and imaginary parts, "SoA"):
//   - the eq tables E1 = eq(r1, .), E2 = eq(r2, .) and EQ(x) = E1 E2;
//   - the bound sides of the product (an integer table bound at a point of
//     F_{p^2} is the pair of its F_p bindings with the eq table's two parts,
//     so the F_p binding kernels serve);
//   - the plane rounds' Gram matrix G = sum_x EQ(x) bit bit^T, whose two
//     parts the F_p Gram pass computes from EQ's two parts;
//   - every folded table of the rounds.
// Rounds run one launch per round (a pass over the pairs that evaluates the
// round polynomial and folds the tables in place) while the tables are
// large, and the last rounds of an instance in one workgroup over LDS; this
// is slower than the F_p path's fused passes.
#include "common.hpp"
#include "m61.hpp"
#include "gram_reduce.hpp"
#include "fs_device.hpp"
#include "sha256.hpp"

namespace ra {

struct f2 {
    uint64_t re, im;
};

__device__ __forceinline__ f2 f2of(uint64_t a) { return f2{a, 0}; }
__device__ __forceinline__ f2 f2add(f2 a, f2 b) { return f2{m61::add(a.re, b.re), m61::add(a.im, b.im)}; }
__device__ __forceinline__ f2 f2sub(f2 a, f2 b) { return f2{m61::sub(a.re, b.re), m61::sub(a.im, b.im)}; }
// (a0 + a1 i)(b0 + b1 i) = (a0 b0 - a1 b1) + ((a0 + a1)(b0 + b1) - a0 b0 - a1 b1) i:
// three products of F_p instead of four
__device__ __forceinline__ f2 f2mul(f2 a, f2 b)
{
    const uint64_t p0 = m61::mul(a.re, b.re), p1 = m61::mul(a.im, b.im);
    const uint64_t p2 = m61::mul(m61::add(a.re, a.im), m61::add(b.re, b.im));
    return f2{m61::sub(p0, p1), m61::sub(m61::sub(p2, p0), p1)};
}
// a c for a small integer c (|c| < 2^31)
__device__ __forceinline__ f2 f2small(f2 a, int32_t c) { return f2{m61::mul_small(a.re, c), m61::mul_small(a.im, c)}; }
// a c for an F_p element c
__device__ __forceinline__ f2 f2scale(f2 a, uint64_t c) { return f2{m61::mul(a.re, c), m61::mul(a.im, c)}; }
__device__ __forceinline__ f2 ldp(const uint64_t *p) { return f2{p[0], p[1]}; }  // a challenge (re, im)
__device__ __forceinline__ void stp(uint64_t *p, f2 v)
{
    p[0] = v.re;
    p[1] = v.im;
}
__device__ __forceinline__ f2 ldt(const F2Tab &t, uint64_t i) { return f2{t.re[i], t.im[i]}; }
__device__ __forceinline__ void stt(const F2Tab &t, uint64_t i, f2 v)
{
    t.re[i] = v.re;
    t.im[i] = v.im;
}
// eq(z, b) for one variable and a bit b
__device__ __forceinline__ f2 eq1b(f2 z, int b) { return b ? z : f2sub(f2of(1), z); }
// eq(z, X) = (1 - X) + z (2 X - 1) for a small integer X
__device__ __forceinline__ f2 eq1x(f2 z, int X) { return f2add(f2of(m61::from_i64(1 - X)), f2small(z, 2 * X - 1)); }

// Block sum of the eight words of four F_{p^2} values; thread 0 writes them.
__device__ __forceinline__ void f2_block_out(const f2 (&acc)[4], uint64_t *red, uint64_t *out)
{
    uint64_t v[8];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        v[2 * q] = acc[q].re;
        v[2 * q + 1] = acc[q].im;
    }
    m61::block_sum<8>(v, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int q = 0; q < 8; q++) out[q] = v[q];
}

// ---------------------------------------------------------------------------
// eq tables (Eq. (1)) of points of F_{p^2}: the point is v challenges stored
// as pairs (re, im); the table goes to two F_p arrays.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_f2_eq(const uint64_t *__restrict__ z, int v, F2Tab out)
{
    __shared__ f2 zl[64];
    if ((int)threadIdx.x < v) zl[threadIdx.x] = ldp(z + 2 * threadIdx.x);
    __syncthreads();
    const uint64_t n = 1ull << v;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x) {
        f2 acc = f2of(1);
        for (int j = 0; j < v; j++) acc = f2mul(acc, eq1b(zl[j], (int)((i >> (v - 1 - j)) & 1)));
        stt(out, i, acc);
    }
}

void launch_f2_eq(const uint64_t *z, int v, F2Tab out, hipStream_t st)
{
    const uint64_t n = 1ull << v;
    const int nb = (int)((n + kThreads - 1) / kThreads < 1024 ? (n + kThreads - 1) / kThreads : 1024);
    hipLaunchKernelGGL(k_f2_eq, dim3(nb), dim3(kThreads), 0, st, z, v, out);
}

// EQ(x) = E1[x >> lk] E2[x mod 2^lk] for x < N (the eq table of (r1, r2)).
__global__ __launch_bounds__(256) void k_f2_outer(F2Tab E1, F2Tab E2, int lk, uint64_t N, F2Tab out)
{
    const uint64_t mask = (1ull << lk) - 1;
    for (uint64_t x = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < N; x += (uint64_t)gridDim.x * blockDim.x)
        stt(out, x, f2mul(ldt(E1, x >> lk), ldt(E2, x & mask)));
}

void launch_f2_outer(F2Tab E1, F2Tab E2, int lk, uint64_t N, F2Tab out, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_outer, dim3(f2_blocks(N)), dim3(kThreads), 0, st, E1, E2, lk, N, out);
}

// The claims R~, Rm~, Y~, Z~ at (r1, r2): sum_x EQ(x) v(x), per-block
// partials (eight words per block).
__global__ __launch_bounds__(256) void k_f2_claims(F2Tab EQ, const int32_t *__restrict__ R,
                                                   const uint16_t *__restrict__ Rm, const int32_t *__restrict__ Y,
                                                   const int32_t *__restrict__ Z, uint64_t N, uint64_t *part)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    f2 acc[4] = {f2of(0), f2of(0), f2of(0), f2of(0)};
    for (uint64_t x = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < N; x += (uint64_t)gridDim.x * blockDim.x) {
        const f2 e = ldt(EQ, x);
        acc[0] = f2add(acc[0], f2small(e, R[x]));
        acc[1] = f2add(acc[1], f2small(e, (int32_t)Rm[x]));
        acc[2] = f2add(acc[2], f2small(e, Y[x]));
        acc[3] = f2add(acc[3], f2small(e, Z[x]));
    }
    f2_block_out(acc, red, part + 8 * (size_t)blockIdx.x);
}

void launch_f2_claims(F2Tab EQ, const int32_t *R, const uint16_t *Rm, const int32_t *Y, const int32_t *Z, uint64_t N,
                      uint64_t *part, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_claims, dim3(f2_blocks(N)), dim3(kThreads), 0, st, EQ, R, Rm, Y, Z, N, part);
}

// Sum of nb rows of eight partial words -> out[0..7].
__global__ __launch_bounds__(256) void k_f2_sum8(const uint64_t *__restrict__ part, int nb, uint64_t *out)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    uint64_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int b = threadIdx.x; b < nb; b += blockDim.x)
#pragma unroll
        for (int q = 0; q < 8; q++) v[q] = m61::add(v[q], part[8 * (size_t)b + q]);
    m61::block_sum<8>(v, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int q = 0; q < 8; q++) out[q] = v[q];
}

void launch_f2_sum8(const uint64_t *part, int nb, uint64_t *out, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_sum8, dim3(1), dim3(kThreads), 0, st, part, nb, out);
}

// ---------------------------------------------------------------------------
// One round of a sum-check instance over tables of 2h entries (Sec. II-D):
// for every pair (i, i + h) the summand at X = 0..3 (each table is lo +
// X (hi - lo) there), summed per block, and the fold T[i] <- lo + rho
// (hi - lo) into the destination tables.  Summands:
//   F2_MATMUL  a b                                  (tables a, b; degree 2)
//   F2_RANGE   EQ B (c_eq (B - 1) + c_w)            (tables EQ, B; degree 3),
//              the range summand once the plane variables are bound:
//              c_eq = eq(tau_p, sigma_p), c_w = mu W~(sigma_p)
//   F2_RELU    EQ D S, D = R - Y, S = R + Y         (Eq. (6); degree 3)
// The first round of the ReLU instance reads R, Y (int32) for D, S.
// ---------------------------------------------------------------------------
// The summand of one pair at X = 0..3 added into acc, and the folded values
// lo + rho (hi - lo) into lo.
template <int KIND>
__device__ __forceinline__ void f2_pair(f2 (&lo)[3], const f2 (&hi)[3], f2 rho, f2 ceq, f2 cw, f2 (&acc)[4])
{
    constexpr int NT = KIND == F2_RELU ? 3 : 2;
    f2 v[3], d[3];
#pragma unroll
    for (int q = 0; q < NT; q++) {
        v[q] = lo[q];
        d[q] = f2sub(hi[q], lo[q]);
    }
#pragma unroll
    for (int X = 0; X < 4; X++) {
        if (X > 0)
#pragma unroll
            for (int q = 0; q < NT; q++) v[q] = f2add(v[q], d[q]);  // the tables at X
        f2 f;
        if (KIND == F2_MATMUL) {
            if (X == 3) break;
            f = f2mul(v[0], v[1]);
        } else if (KIND == F2_RANGE) {
            f = f2mul(f2mul(v[0], v[1]), f2add(f2mul(ceq, f2sub(v[1], f2of(1))), cw));
        } else {
            f = f2mul(f2mul(v[0], v[1]), v[2]);
        }
        acc[X] = f2add(acc[X], f);
    }
#pragma unroll
    for (int q = 0; q < NT; q++) lo[q] = f2add(lo[q], f2mul(rho, d[q]));
}

// The ReLU instance's first round reads D = R - Y and S = R + Y from the
// integer tables.
__device__ __forceinline__ void f2_relu_ints(const int32_t *R, const int32_t *Y, uint64_t i, f2 &d, f2 &s)
{
    const int64_t r = R[i], y = Y[i];
    d = f2of(m61::from_i64(r - y));
    s = f2of(m61::from_i64(r + y));
}

template <int KIND>
__global__ __launch_bounds__(256) void k_f2_round(F2RoundArgs a)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    constexpr int NT = KIND == F2_RELU ? 3 : 2;
    const f2 rho = ldp(a.rho);
    f2 ceq = f2of(0), cw = f2of(0);
    if (KIND == F2_RANGE) {
        ceq = ldp(a.cst);
        cw = ldp(a.cst + 2);
    }
    f2 acc[4] = {f2of(0), f2of(0), f2of(0), f2of(0)};
    const uint64_t h = a.h;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < h; i += (uint64_t)gridDim.x * blockDim.x) {
        f2 lo[3], hi[3];
        lo[0] = ldt(a.src[0], i);
        hi[0] = ldt(a.src[0], i + h);
        if (KIND == F2_RELU && a.first) {
            f2_relu_ints(a.R, a.Y, i, lo[1], lo[2]);
            f2_relu_ints(a.R, a.Y, i + h, hi[1], hi[2]);
        } else {
#pragma unroll
            for (int q = 1; q < NT; q++) {
                lo[q] = ldt(a.src[q], i);
                hi[q] = ldt(a.src[q], i + h);
            }
        }
        f2_pair<KIND>(lo, hi, rho, ceq, cw, acc);
#pragma unroll
        for (int q = 0; q < NT; q++) stt(a.dst[q], i, lo[q]);
    }
    f2_block_out(acc, red, a.part + 8 * (size_t)blockIdx.x);
}

// ---------------------------------------------------------------------------
// The last v <= kF2TailLog rounds of an instance in one workgroup: the tables
// (2^v entries) are staged in LDS and folded there, round after round; each
// round's sums go to its first partial slot (the round's other slots are
// zeroed, so the finish kernel reads the same layout as after k_f2_round),
// and the final values to index 0 of the destination tables.
// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(256) void k_f2_tail(F2TailArgs a)
{
    constexpr int NT = KIND == F2_RELU ? 3 : 2, S = 1 << kF2TailLog;
    __shared__ uint64_t T[NT][2][S];  // (re, im) of each table
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    __shared__ uint64_t rz[2 * kF2TailLog];
    const int tid = threadIdx.x, n0 = 1 << a.v;
    f2 ceq = f2of(0), cw = f2of(0);
    if (KIND == F2_RANGE) {
        ceq = ldp(a.cst);
        cw = ldp(a.cst + 2);
    }
    if (tid < 2 * a.v) rz[tid] = a.rho[tid];
    for (int i = tid; i < n0; i += blockDim.x) {
        f2 t[3];
        t[0] = ldt(a.src[0], i);
        if (KIND == F2_RELU && a.first) {
            f2_relu_ints(a.R, a.Y, i, t[1], t[2]);
        } else {
#pragma unroll
            for (int q = 1; q < NT; q++) t[q] = ldt(a.src[q], i);
        }
#pragma unroll
        for (int q = 0; q < NT; q++) {
            T[q][0][i] = t[q].re;
            T[q][1][i] = t[q].im;
        }
    }
    __syncthreads();
    for (int c = 0; c < a.v; c++) {
        const int h = n0 >> (c + 1);
        const f2 rho{rz[2 * c], rz[2 * c + 1]};
        f2 acc[4] = {f2of(0), f2of(0), f2of(0), f2of(0)};
        // a pair's entries are read and its fold written by one thread only
        for (int i = tid; i < h; i += blockDim.x) {
            f2 lo[3], hi[3];
#pragma unroll
            for (int q = 0; q < NT; q++) {
                lo[q] = f2{T[q][0][i], T[q][1][i]};
                hi[q] = f2{T[q][0][i + h], T[q][1][i + h]};
            }
            f2_pair<KIND>(lo, hi, rho, ceq, cw, acc);
#pragma unroll
            for (int q = 0; q < NT; q++) {
                T[q][0][i] = lo[q].re;
                T[q][1][i] = lo[q].im;
            }
        }
        uint64_t *part = a.part + (size_t)c * kF2MaxBlocks * 8;
        const int nb = f2_blocks((uint64_t)h);
        if (tid >= 1 && tid < nb)
#pragma unroll
            for (int q = 0; q < 8; q++) part[8 * tid + q] = 0;
        f2_block_out(acc, red, part);  // its barriers also order this round's folds before the next reads
        __syncthreads();
    }
    if (tid == 0)
#pragma unroll
        for (int q = 0; q < NT; q++) stt(a.dst[q], 0, f2{T[q][0][0], T[q][1][0]});
}

void launch_f2_tail(const F2TailArgs &a, hipStream_t st)
{
    switch (a.kind) {
    case F2_MATMUL: hipLaunchKernelGGL(k_f2_tail<F2_MATMUL>, dim3(1), dim3(kThreads), 0, st, a); break;
    case F2_RANGE: hipLaunchKernelGGL(k_f2_tail<F2_RANGE>, dim3(1), dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL(k_f2_tail<F2_RELU>, dim3(1), dim3(kThreads), 0, st, a); break;
    }
}

void launch_f2_round(const F2RoundArgs &a, hipStream_t st)
{
    const dim3 grid(f2_blocks(a.h));
    switch (a.kind) {
    case F2_MATMUL: hipLaunchKernelGGL(k_f2_round<F2_MATMUL>, grid, dim3(kThreads), 0, st, a); break;
    case F2_RANGE: hipLaunchKernelGGL(k_f2_round<F2_RANGE>, grid, dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL(k_f2_round<F2_RELU>, grid, dim3(kThreads), 0, st, a); break;
    }
}

// ---------------------------------------------------------------------------
// The rounds' evaluations from the blocks' partials (one workgroup per
// round: round j of an instance over 2^v entries had f2_blocks(2^(v-1-j))
// blocks), written as pairs, D + 1 per round; workgroup 0 also writes the
// instance's final words:
//   F2_MATMUL  c0 = g_1(0) + g_1(1) (a b with no rounds), a*, b*
//   F2_RANGE   b~(sigma)
//   F2_RELU    R~(rho') = (D + S) / 2, Y~(rho') = (S - D) / 2
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_f2_finish(F2FinishArgs a)
{
    __shared__ uint64_t red[m61::block_sum_words(8, 256)];
    const int j = blockIdx.x, D = a.kind == F2_MATMUL ? 2 : 3;
    uint64_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (j < a.v) {
        const int nb = f2_blocks(1ull << (a.v - 1 - j));
        const uint64_t *p = a.part + (size_t)j * kF2MaxBlocks * 8;
        for (int b = threadIdx.x; b < nb; b += blockDim.x)
#pragma unroll
            for (int q = 0; q < 8; q++) v[q] = m61::add(v[q], p[8 * (size_t)b + q]);
        m61::block_sum<8>(v, red);
        if (threadIdx.x == 0)
            for (int q = 0; q < 2 * (D + 1); q++) a.ev[2 * (D + 1) * j + q] = v[q];
    }
    if (j != 0 || threadIdx.x != 0) return;
    if (a.kind == F2_MATMUL) {
        const f2 t0 = ldt(a.t[0], 0), t1 = ldt(a.t[1], 0);
        const f2 c0 = a.v > 0 ? f2add(f2{v[0], v[1]}, f2{v[2], v[3]}) : f2mul(t0, t1);
        stp(a.fin, c0);
        stp(a.fin + 2, t0);
        stp(a.fin + 4, t1);
    } else if (a.kind == F2_RANGE) {
        stp(a.fin, ldt(a.t[1], 0));
    } else {
        f2 Dv, Sv;
        if (a.v > 0) {
            Dv = ldt(a.t[1], 0);
            Sv = ldt(a.t[2], 0);
        } else {
            Dv = f2of(m61::from_i64((int64_t)a.R[0] - a.Y[0]));
            Sv = f2of(m61::from_i64((int64_t)a.R[0] + a.Y[0]));
        }
        constexpr uint64_t inv2 = 1ull << 60;  // 2 2^60 = 2^61 = 1 mod p
        stp(a.fin, f2scale(f2add(Dv, Sv), inv2));
        stp(a.fin + 2, f2scale(f2sub(Sv, Dv), inv2));
    }
}

void launch_f2_finish(const F2FinishArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_finish, dim3(a.v > 0 ? a.v : 1), dim3(kThreads), 0, st, a);
}

// ---------------------------------------------------------------------------
// The plane rounds of the range instance from the Gram matrix (one
// workgroup).  With the plane variables q_1 .. q_{j-1} bound to sigma and q_j
// = X, the table is b(sigma_<j, X, q', x) = sum_{y, z} c_X(y, z)
// bit_{(y, z, q')}(x) with c_X(y, z) = eq(sigma_<j, y) eq(X, z), so
//   g_j(X) = sum_{q'} E(X, q') (Q - L) + mu Wt(X, q') L,
//   Q = c^T G c, L = sum c G_diag (a bit squared is itself),
//   E(X, q') = eq(tau_p, (sigma_<j, X, q')), Wt(X, q') = W~(sigma_<j, X, q'),
// where the sums run over the planes (y, z, q') and G[p][p'] = sum_x EQ(x)
// bit_p(x) bit_p'(x).  Also writes the x rounds' constants c_eq =
// eq(tau_p, sigma_p), c_w = mu W~(sigma_p) and the claimed sum
// mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~).  G and the challenges are staged
// in LDS.  Round j has 4 P / 2^(j+1) items (X, q') of 2^(j+1) rows each, so
// 4 P <= 256 threads take one (item, row) pair each; an item's rows are
// adjacent lanes and are summed by a butterfly inside their lane group.
// ---------------------------------------------------------------------------
// eq(a, b) for one variable, both points in F_{p^2}: a b + (1 - a)(1 - b)
__device__ __forceinline__ f2 eq1z(f2 a, f2 b) { return f2add(f2mul(a, b), f2mul(f2sub(f2of(1), a), f2sub(f2of(1), b))); }

__device__ __forceinline__ f2 group_sum(f2 v, int width)
{
    for (int off = 1; off < width; off <<= 1)
        v = f2{m61::add(v.re, __shfl_xor(v.re, off, 64)), m61::add(v.im, __shfl_xor(v.im, off, 64))};
    return v;
}

__global__ __launch_bounds__(256) void k_f2_planes(F2PlaneArgs a)
{
    constexpr int GS = 65;  // row stride of the staged Gram matrix (odd, so rows start in different banks)
    __shared__ uint64_t g_re[64 * GS], g_im[64 * GS];
    __shared__ f2 W[64], cpre[32], contrib[4][32], tau[8], sig[8], lam[4], pre[8], gsh[4];
    __shared__ uint32_t fsbuf32[kFsLdsBytes / 4];  // the transcript (Fiat-Shamir mode)
    uint8_t *fsbuf = (uint8_t *)fsbuf32;
    const int tid = threadIdx.x, lP = a.lP, P = a.P;
    for (int e = tid; e < P * P; e += blockDim.x) {
        const int p = e >> lP, q = e & (P - 1);
        g_re[p * GS + q] = a.G_re[p * 64 + q];
        g_im[p * GS + q] = a.G_im[p * 64 + q];
    }
    if (tid < lP) {
        tau[tid] = ldp(a.tau + 2 * tid);
        if (!a.fs) sig[tid] = ldp(a.sig + 2 * tid);  // else drawn after each round
    }
    if (tid < 4) lam[tid] = ldp(a.lam + 2 * tid);
    __syncthreads();
    const f2 mu = lam[3];
    if (tid < 64) {
        f2 w = f2of(0);
        const int s = a.s, t = a.t;
        if (tid < s) w = f2scale(lam[0], 1ull << tid);
        else if (tid < s + t + 2) w = f2scale(lam[1], 1ull << (tid - s));
        else if (a.relu && tid < s + 2 * t + 4) w = f2scale(lam[2], 1ull << (tid - s - t - 2));
        W[tid] = tid < P ? w : f2of(0);
    }
    if (tid == 0) {
        pre[0] = f2of(1);  // pre[i] = prod over i' < i of eq(tau_i', sigma_i'), after round i - 1
        if (a.fs) fs_pull(a.fs, fsbuf);
    }
    for (int jj = 0; jj < lP; jj++) {
        __syncthreads();
        if (tid < (1 << jj)) {
            f2 c = f2of(1);
            for (int i = 0; i < jj; i++) c = f2mul(c, eq1b(sig[i], (tid >> (jj - 1 - i)) & 1));
            cpre[tid] = c;
        }
        __syncthreads();
        const int sh = lP - jj - 1, nq = 1 << sh, nrows = 2 << jj;
        const int item = tid >> (jj + 1), r = tid & (nrows - 1);
        const int X = item >> sh, qp = item & (nq - 1);
        const bool on = tid < 4 * P;
        auto coef = [&](int row) {
            const f2 c = cpre[row >> 1];
            return (row & 1) ? f2small(c, X) : f2small(c, 1 - X);
        };
        f2 Q = f2of(0), L = f2of(0), Ws = f2of(0);
        if (on) {
            const int pr = (r << sh) | qp;
            const uint64_t *gr = g_re + pr * GS + qp, *gi = g_im + pr * GS + qp;
            // four independent partial sums, so the products of four rows are
            // in flight together (the sum is exact in any order)
            f2 r4[4] = {f2of(0), f2of(0), f2of(0), f2of(0)};
            int c = 0;
            for (; c + 3 < nrows; c += 4)
#pragma unroll
                for (int u = 0; u < 4; u++)
                    r4[u] = f2add(r4[u], f2mul(coef(c + u), f2{gr[(c + u) << sh], gi[(c + u) << sh]}));
            for (; c < nrows; c++) r4[0] = f2add(r4[0], f2mul(coef(c), f2{gr[c << sh], gi[c << sh]}));
            const f2 row = f2add(f2add(r4[0], r4[1]), f2add(r4[2], r4[3]));
            const f2 cr = coef(r);
            Q = f2mul(cr, row);
            L = f2mul(cr, f2{g_re[pr * GS + pr], g_im[pr * GS + pr]});
            Ws = f2mul(cr, W[pr]);
        }
        Q = group_sum(Q, nrows);
        L = group_sum(L, nrows);
        Ws = group_sum(Ws, nrows);
        if (on && r == 0) {
            f2 E = f2mul(pre[jj], eq1x(tau[jj], X));
            for (int i = jj + 1; i < lP; i++) E = f2mul(E, eq1b(tau[i], (qp >> (lP - 1 - i)) & 1));
            contrib[X][qp] = f2add(f2mul(E, f2sub(Q, L)), f2mul(mu, f2mul(Ws, L)));
        }
        __syncthreads();
        if (tid < 4) {
            f2 g = f2of(0);
            for (int q = 0; q < nq; q++) g = f2add(g, contrib[tid][q]);
            stp(a.ev + 8 * jj + 2 * tid, g);
            gsh[tid] = g;
        }
        __syncthreads();
        if (tid == 0) {
            if (a.fs) {  // the round's values absorbed, sigma_jj drawn
                uint64_t w[8], c[2];
                for (int q = 0; q < 4; q++) {
                    w[2 * q] = gsh[q].re;
                    w[2 * q + 1] = gsh[q].im;
                }
                if (!fs_absorb_words_lds(fsbuf, w, 8)) *a.err = 1;
                fs_draw_lds(fsbuf, c);
                if (jj == lP - 1) fs_push(a.fs, fsbuf);
                sig[jj] = f2{c[0], c[1]};
                stp(a.sig_out + 2 * jj, sig[jj]);
            }
            pre[jj + 1] = f2mul(pre[jj], eq1z(tau[jj], sig[jj]));
        }
    }
    __syncthreads();
    // x rounds' constants and the claimed sum
    if (tid < 64) {
        f2 term = f2of(0);
        if (tid < P) {
            f2 e = f2of(1);
            for (int i = 0; i < lP; i++) e = f2mul(e, eq1b(sig[i], (tid >> (lP - 1 - i)) & 1));
            term = f2mul(e, W[tid]);
        }
        const f2 wsig = f2{m61::wave_sum(term.re), m61::wave_sum(term.im)};
        if (tid == 0) {
            stp(a.cst, pre[lP]);
            stp(a.cst + 2, f2mul(mu, wsig));
            const f2 r = ldp(a.claims), rm = ldp(a.claims + 2), y = ldp(a.claims + 4);
            f2 H = f2add(f2mul(lam[0], rm), f2mul(lam[1], f2add(r, f2of(1ull << (a.t + 1)))));
            if (a.relu) H = f2add(H, f2mul(lam[2], y));
            stp(a.range_sum, f2mul(mu, H));
        }
    }
}

void launch_f2_planes(const F2PlaneArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_planes, dim3(1), dim3(kThreads), 0, st, a);
}

// The Gram matrix from the partial tiles of one Gram pass.
__global__ __launch_bounds__(256) void k_f2_gram_sum(const uint64_t *__restrict__ gpart, int nblk, int tiles,
                                                     uint64_t *__restrict__ G)
{
    __shared__ uint64_t red[kGramReduceLdsWords];
    gram_reduce_block(gpart, nblk, tiles, G, blockIdx.x, red);
}

void launch_f2_gram_sum(const uint64_t *gpart, int nblk, int tiles, uint64_t *G, hipStream_t st)
{
    hipLaunchKernelGGL(k_f2_gram_sum, dim3(gram_reduce_groups(tiles)), dim3(kThreads), 0, st, gpart, nblk, tiles, G);
}

}  // namespace ra
