// xrounds.hip -- the rounds over x of the concatenated range check and of
// the ReLU zero-check (Sec. III-B, Eq. (6)), after the plane variables of
// the range check are bound.  Both instances sum over the same Boolean cube
// with the same equality factor EQ(x) = eq(r, x), r = (r1, r2):
//   range  sum_x EQ(x) (Ep Bx(x)^2 + c Bx(x))          (Bx: bit table bound at sigma_p)
//   ReLU   sum_x EQ(x) (R(x)^2 - Y(x)^2) = sum_x EQ(x) D(x) S(x),   D = R - Y, S = R + Y.
// The range instance binds x to sigma_x, the ReLU instance to rho'.
//
// EQ is never stored.  With x bound to z_<j in round j it equals
//   K_j eq1(r_j, X) eq(r_>j, i),      K_j = prod_{l<j} eq1(r_l, z_l),
// so the round polynomial is K_j eq1(r_j, X) s_j(X) with
//   s_j(X) = sum_i eq(r_>j, i) h(T_X(i))     (T_X = T_lo + X (T_hi - T_lo)),
// a quadratic in X.  The kernels accumulate, per round, with w_i = eq(r_>j, i),
//   range  A_a = sum_i w_i b_a (a = 0, 1),  Q_a = sum_i w_i b_a^2 (a = 0, 1),  M = sum_i w_i b_0 b_1
//   ReLU   Z_a = sum_i w_i d_a s_a (a = 0, 1),  U = sum_i w_i (d_0 + d_1)(s_0 + s_1)
// five products per pair and instance.  The values at X = 2 follow from
// b_2 = 2 b_1 - b_0 (and likewise d_2, s_2):
//   A_2 = 2 A_1 - A_0,  Q_2 = Q_0 + 4 (Q_1 - M),  Z_2 = 3 Z_0 + 6 Z_1 - 2 U;
// the assembly forms s_j(0..2), extrapolates s_j(3) and multiplies by
// K_j eq1(r_j, X).  The weights eq(r_>j, i) come from two small tables of
// suffix eq vectors (a high part and a low part of the variables), so they
// cost one product per thread.  The ReLU tables are kept as D and S; the
// final values give R = (D + S) / 2 and Y = (S - D) / 2.
//
// Arithmetic inside the kernels uses loose residues (m61.hpp): products and
// differences are folded below 2^61 + 8 without a final comparison, sums of
// at most four folded terms are added to a folded accumulator before it is
// folded again, and every value leaving a kernel is canonical.
#include <algorithm>

#include "assemble.hpp"
#include "common.hpp"
#include "m61.hpp"
#include "plane_round.hpp"

namespace ra {

// Terms of one pair with weight w, added to acc without folding (each term
// is a folded value): range acc[0..5) = A_0, A_1, Q_0, Q_1, M; ReLU
// acc[0..3) = Z_0, Z_1, U.  Inputs are folded or canonical.
__device__ __forceinline__ void range_pair(uint64_t w, uint64_t b0, uint64_t b1, uint64_t *acc)
{
    const uint64_t eb0 = m61::lmul(w, b0), eb1 = m61::lmul(w, b1);
    acc[0] += eb0;
    acc[1] += eb1;
    acc[2] += m61::lmul(eb0, b0);
    acc[3] += m61::lmul(eb1, b1);
    acc[4] += m61::lmul(eb0, b1);
}

__device__ __forceinline__ void relu_pair(uint64_t w, uint64_t d0, uint64_t d1, uint64_t s0, uint64_t s1,
                                          uint64_t *acc)
{
    const uint64_t ed0 = m61::lmul(w, d0), ed1 = m61::lmul(w, d1);
    acc[0] += m61::lmul(ed0, s0);
    acc[1] += m61::lmul(ed1, s1);
    acc[2] += m61::lmul(ed0 + ed1, s0 + s1);  // sums of two folded values are loose
}

template <int NV>
__device__ __forceinline__ void fold_all(uint64_t *acc)
{
#pragma unroll
    for (int q = 0; q < NV; q++) acc[q] = m61::fold(acc[q]);
}

// lo + z (hi - lo), folded.
__device__ __forceinline__ uint64_t fold(uint64_t lo, uint64_t hi, uint64_t z)
{
    return m61::fold(lo + m61::lmul(z, m61::lsub(hi, lo)));
}

// Field value of a small signed integer (|v| < 2^62), folded.
__device__ __forceinline__ uint64_t small_to_field(int64_t v) { return m61::fold((uint64_t)v + 4 * m61::P); }

// Sums of NV values over the 64 lanes of the calling wave, written to
// out[0 .. NV).  Every wave of the block calls it at the same point (it holds
// a block barrier); `lw` is the wave's own NV * 68 words of LDS.
template <int NV>
__device__ __forceinline__ void wave_sums_to(const uint64_t (&v)[NV], uint64_t *lw, uint64_t *out)
{
    constexpr int LS = 68;  // padded stride: 16 lanes read 16 distinct bank pairs
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < NV; q++) lw[q * LS + lane] = v[q];
    __syncthreads();
    for (int t = lane; t < 4 * NV; t += 64) {  // four lanes per value, 16 entries each
        const uint64_t *src = lw + (t >> 2) * LS + (t & 3);
        uint64_t a0 = 0, a1 = 0;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            a0 = m61::add(a0, src[4 * e]);
            a1 = m61::add(a1, src[4 * e + 4]);
        }
        uint64_t sum = m61::add(a0, a1);
        sum = m61::add(sum, __shfl_xor(sum, 1, 64));
        sum = m61::add(sum, __shfl_xor(sum, 2, 64));
        if ((t & 3) == 0) out[t >> 2] = sum;
    }
}

// ---------------------------------------------------------------------------
// C fused rounds j .. j + C - 1 over tables of S = 2^lS entries (lS = lN - j).
// Sub-cube i (< S' = S / 2^C) is the set of entries i + t S' (t < 2^C), the
// values of the C variables being bound; one thread runs the C rounds on one
// sub-cube in registers and writes the bound value to index i.  The pair
// (u, u + h) of local round c has weight eq(r_{j+c+1 .. j+C-1}, u)
// eq(r_{j+C ..}, i), built from eq(r_{j+C ..}, i) = HS[.] LS[.] by halving.
// With ReLU, waves 0-1 of a block run the range instance and waves 2-3 the
// ReLU instance on the same 128 sub-cubes (so a wave carries half the work);
// without, all four waves run the range instance.  With FIRST the inputs are
// Bx and the integer R, Y; D and S are written.  Each wave writes its sums
// of round c to part + c * stride + 8 unit (range words 0-4, ReLU 5-7).
// ---------------------------------------------------------------------------
template <int C>
__device__ __forceinline__ void x_weights(uint64_t e, const uint64_t *rr, uint64_t (&w)[1 << C])
{
    // round c uses w[(1 << (C-1-c)) - 1 + u] (indices 0 .. 2^C - 2)
    w[0] = e;  // round C - 1 (u empty)
#pragma unroll
    for (int c = C - 2; c >= 0; c--) {
        const int hn = 1 << (C - 1 - c), base = hn - 1, pb = (hn >> 1) - 1;
        // u = (msb, rest): eq1(r_{j+c+1}, msb) times the weight of `rest` one round later
#pragma unroll
        for (int u = 0; u < hn / 2; u++) {
            const uint64_t hi = m61::lmul(rr[c + 1], w[pb + u]);
            w[base + hn / 2 + u] = hi;
            w[base + u] = m61::lsub(w[pb + u], hi);
        }
    }
}

// The sub-cubes of one thread for one instance (ZW: ReLU, else range); the
// sums of round c are added to acc[c] (folded values).
// eq(r_{lN-nvar .. lN-1}, k) from the suffix heaps (folded or canonical).
__device__ __forceinline__ uint64_t suffix_weight(const uint64_t *HS, const uint64_t *LS, int nvar, int L, uint64_t k)
{
    if (nvar <= L) return LS[(1ull << nvar) + k];
    return m61::lmul(HS[(1ull << (nvar - L)) + (k >> L)], LS[(1ull << L) + (k & ((1ull << L) - 1))]);
}

// Extra workgroup q of an x-round launch (256 threads): assemble a slot of
// the launch before, or evaluate a plane round.
__device__ __forceinline__ void x_job(const XJobs &jobs, int q, uint64_t *lds)
{
    if (q < jobs.nslot) assemble_slot(jobs.s[q], jobs.part + (size_t)q * jobs.stride, jobs.tr, jobs.xc, lds);
    else if (q - jobs.nslot < jobs.nplane) plane_round(jobs.pa, q - jobs.nslot + 1, lds);
}

// The sub-cubes of one thread for one instance (ZW: ReLU, else range); the
// sums of round c are added to acc[c] (folded values).
template <int C, bool FIRST, bool ZW>
__device__ __forceinline__ void x_sub_cubes(const XArgs &a, uint64_t sub, uint64_t i0, uint64_t step,
                                            uint64_t (&acc)[C][ZW ? 3 : 5])
{
    constexpr int NL = 1 << C, NV = ZW ? 3 : 5;
#pragma unroll
    for (int c = 0; c < C; c++)
#pragma unroll
        for (int q = 0; q < NV; q++) acc[c][q] = 0;
    uint64_t rz[C], rr[C];
#pragma unroll
    for (int c = 0; c < C; c++) {
        rz[c] = ZW ? a.rho_z[c] : a.rho_a[c];
        rr[c] = a.r[a.j + c];
    }
    const int nvar = a.lN - a.j - C;
    for (uint64_t i = i0; i < sub; i += step) {
        uint64_t w[NL];
        x_weights<C>(suffix_weight(a.HS, a.LS, nvar, a.L, i), rr, w);
        if (!ZW) {
            uint64_t b[NL];
#pragma unroll
            for (int t = 0; t < NL; t++) b[t] = a.bx[i + t * sub];
#pragma unroll
            for (int c = 0; c < C; c++) {
                const int h = NL >> (c + 1), base = h - 1;
#pragma unroll
                for (int u = 0; u < h; u++) {
                    range_pair(w[base + u], b[u], b[u + h], acc[c]);
                    b[u] = fold(b[u], b[u + h], rz[c]);
                    if ((u & 3) == 3 || u == h - 1) fold_all<NV>(acc[c]);
                }
            }
            a.bx[i] = m61::canon(b[0]);
        } else {
            uint64_t d[NL], s[NL];
#pragma unroll
            for (int t = 0; t < NL; t++) {
                if (FIRST) {
                    const int64_t R = a.R[i + t * sub], Y = a.Y[i + t * sub];
                    d[t] = small_to_field(R - Y);
                    s[t] = small_to_field(R + Y);
                } else {
                    d[t] = a.d[i + t * sub];
                    s[t] = a.s[i + t * sub];
                }
            }
#pragma unroll
            for (int c = 0; c < C; c++) {
                const int h = NL >> (c + 1), base = h - 1;
#pragma unroll
                for (int u = 0; u < h; u++) {
                    relu_pair(w[base + u], d[u], d[u + h], s[u], s[u + h], acc[c]);
                    d[u] = fold(d[u], d[u + h], rz[c]);
                    s[u] = fold(s[u], s[u + h], rz[c]);
                    if ((u & 3) == 3 || u == h - 1) fold_all<NV>(acc[c]);
                }
            }
            a.d[i] = m61::canon(d[0]);
            a.s[i] = m61::canon(s[0]);
        }
    }
}

template <int C>
constexpr int xrounds_lds_words()
{
    return 4 * (5 * C) * 68 + 4 * (5 * C) > kJobLdsWords ? 4 * (5 * C) * 68 + 4 * (5 * C) : kJobLdsWords;
}

// Workgroups below nmain run the rounds; the others are jobs.
template <int C, bool FIRST, bool RELU>
__global__ __launch_bounds__(256) void k_xrounds(XArgs a, uint64_t sub, int stride, XJobs jobs, int nmain)
{
    constexpr int NPB = RELU ? 128 : 256, NVR = 5 * C;
    __shared__ uint64_t smem[xrounds_lds_words<C>()];
    if ((int)blockIdx.x >= nmain) {
        x_job(jobs, blockIdx.x - nmain, smem);
        return;
    }
    uint64_t *tot = smem + 4 * NVR * 68;
    const int tid = threadIdx.x, wv = tid >> 6;
    const bool zw = RELU && wv >= 2;  // wave-uniform
    const int lt = RELU ? (tid & 127) : tid;
    const int unit = RELU ? blockIdx.x * 2 + (wv & 1) : blockIdx.x * 4 + wv;
    const uint64_t i0 = (uint64_t)blockIdx.x * NPB + lt, step = (uint64_t)nmain * NPB;
    // per-wave sums; the range waves' layout covers both (ReLU values in the first 3 C)
    uint64_t flat[NVR];
    if (!zw) {
        uint64_t acc[C][5];
        x_sub_cubes<C, FIRST, false>(a, sub, i0, step, acc);
#pragma unroll
        for (int c = 0; c < C; c++)
#pragma unroll
            for (int q = 0; q < 5; q++) flat[c * 5 + q] = m61::canon(acc[c][q]);
    } else {
        uint64_t acc[C][3];
        x_sub_cubes<C, FIRST, true>(a, sub, i0, step, acc);
#pragma unroll
        for (int c = 0; c < C; c++)
#pragma unroll
            for (int q = 0; q < 5; q++) flat[c * 5 + q] = q < 3 ? m61::canon(acc[c][q]) : 0;
    }
    wave_sums_to<NVR>(flat, smem + wv * NVR * 68, tot + wv * NVR);
    __syncthreads();
    const int lane = tid & 63;
    if (lane < C * 8) {
        const int c = lane >> 3, q = lane & 7;
        uint64_t v;
        if (!zw) v = q < 5 ? tot[wv * NVR + c * 5 + q] : 0;
        else v = tot[wv * NVR + c * 5 + q - 5];
        if (zw ? q >= 5 : (q < 5 || !RELU)) a.part[(size_t)c * stride + (size_t)unit * 8 + q] = v;
    }
}

static int xround_blocks(uint64_t sub, bool relu)
{
    const uint64_t per = relu ? 128 : 256, cap = relu ? kMaxUnits / 2 : kMaxUnits / 4;
    const uint64_t b = (sub + per - 1) / per;
    return (int)(b < cap ? (b ? b : 1) : cap);
}

int xround_units(uint64_t sub, bool relu) { return xround_blocks(sub, relu) * (relu ? 2 : 4); }

void launch_xrounds(int C, bool first, bool relu, const XArgs &a, uint64_t S, int stride, const XJobs &jobs,
                    hipStream_t st)
{
    const uint64_t sub = S >> C;
    const int nmain = xround_blocks(sub, relu);
    const dim3 g(nmain + jobs.nslot + jobs.nplane), b(kThreads);
#define RA_X(CC, F, Z) hipLaunchKernelGGL((k_xrounds<CC, F, Z>), g, b, 0, st, a, sub, stride, jobs, nmain)
#define RA_X_FZ(CC)                      \
    if (first) {                         \
        if (relu) RA_X(CC, true, true);  \
        else RA_X(CC, true, false);      \
    } else {                             \
        if (relu) RA_X(CC, false, true); \
        else RA_X(CC, false, false);     \
    }
    switch (C) {
    case 1: RA_X_FZ(1) break;
    case 2: RA_X_FZ(2) break;
    case 3: RA_X_FZ(3) break;
    default: RA_X_FZ(4) break;
    }
#undef RA_X_FZ
#undef RA_X
}

// ---------------------------------------------------------------------------
// B rounds per workgroup with the sub-cube in LDS.  Workgroup k loads the
// 2^B entries k + t 2^(lS - B) of each table (threads 0-127 the range table,
// 128-255 the ReLU tables D and S; all 256 the range table without ReLU).
// Round c pairs u and u + h (h = 2^(B-1-c)) with weight
//   eq(r_{j+c+1 .. j+B-1}, u) eq(r_{j+B ..}, k) = W[h + u] e_k,
// W the heap of suffix eq tables of the window r_{j+1 .. j+B-1} (set-up: the
// WS heap, or for the last pass the LS heap), e_k from the suffix heaps.  Each thread keeps its sums of a
// round in LDS; at the end the workgroup reduces them per round and either
// writes one partial per round (several sub-cubes) or, for the single
// sub-cube of the last pass, the round polynomials themselves.
// ---------------------------------------------------------------------------
constexpr int kXbMax = 1 << kXBlockMax;
// Thread-rounds (sum over the rounds of min(h, threads per instance)) for
// B <= 10: range 256 + 256 + 255 without ReLU, 128 + 128 + 128 + 127 with it.
constexpr int kXbRoundsR = 767, kXbRoundsZ = 511;
// LDS layout (words): Tb, Td, Ts, W (kXbMax each), challenges (3 x 16), the
// per-thread round sums (range 5, ReLU 3 words), the reduced sums (8 per round).
constexpr int kXbLdsWords = 4 * kXbMax + 48 + 5 * kXbRoundsR + 3 * kXbRoundsZ + 8 * kXBlockMax;
static_assert(kXbLdsWords >= kJobLdsWords, "jobs share the workgroup's LDS");

template <bool RELU>
__global__ __launch_bounds__(256) void k_xblock(XBlockArgs a, int first, XJobs jobs, int nmain)
{
    __shared__ uint64_t smem[kXbLdsWords];
    if ((int)blockIdx.x >= nmain) {
        x_job(jobs, blockIdx.x - nmain, smem);
        return;
    }
    uint64_t *Tb = smem, *Td = Tb + kXbMax, *Ts = Td + kXbMax, *W = Ts + kXbMax;
    uint64_t *rw = W + kXbMax, *za = rw + 16, *zz = za + 16;
    uint64_t *pr = zz + 16, *pz = pr + 5 * kXbRoundsR, *red = pz + 3 * kXbRoundsZ;
    constexpr int NI = RELU ? 128 : 256;  // threads per instance
    const int tid = threadIdx.x, B = a.B, S = 1 << B;
    const bool zw = RELU && tid >= NI;  // wave-uniform
    const int lt = zw ? tid - NI : tid;
    const uint64_t k = blockIdx.x, nsub = 1ull << (a.lS - B);
    // the binding challenges of the B rounds
    if (tid >= 64 && tid < 64 + B) za[tid - 64] = a.rho_a[tid - 64];
    if (RELU && tid >= 128 && tid < 128 + B) zz[tid - 128] = a.rho_z[tid - 128];
    // the sub-cube: at most kXbMax / NI entries per thread, all loads issued first
    constexpr int NQ = kXbMax / NI;
    if (!zw) {
        uint64_t v[NQ];
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const int t = lt + q * NI;
            v[q] = t < S ? a.bx[k + (uint64_t)t * nsub] : 0;
        }
#pragma unroll
        for (int q = 0; q < NQ; q++)
            if (lt + q * NI < S) Tb[lt + q * NI] = v[q];
    } else if (first) {
        int32_t vr[NQ], vy[NQ];
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const int t = lt + q * NI;
            vr[q] = t < S ? a.R[k + (uint64_t)t * nsub] : 0;
            vy[q] = t < S ? a.Y[k + (uint64_t)t * nsub] : 0;
        }
#pragma unroll
        for (int q = 0; q < NQ; q++)
            if (lt + q * NI < S) {
                Td[lt + q * NI] = small_to_field((int64_t)vr[q] - vy[q]);
                Ts[lt + q * NI] = small_to_field((int64_t)vr[q] + vy[q]);
            }
    } else {
        uint64_t vd[NQ], vs[NQ];
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const int t = lt + q * NI;
            vd[q] = t < S ? a.d[k + (uint64_t)t * nsub] : 0;
            vs[q] = t < S ? a.s[k + (uint64_t)t * nsub] : 0;
        }
#pragma unroll
        for (int q = 0; q < NQ; q++)
            if (lt + q * NI < S) {
                Td[lt + q * NI] = vd[q];
                Ts[lt + q * NI] = vs[q];
            }
    }
    // weights W[h + u] e_k of the pairs of every round (W: table s at offset 2^s)
    const uint64_t ek = suffix_weight(a.HS, a.LS, a.lN - a.j - B, a.L, k);
    for (int e0 = tid + 1; e0 < S; e0 += 4 * blockDim.x) {
        uint64_t v[4];
#pragma unroll
        for (int q = 0; q < 4; q++) v[q] = e0 + q * (int)blockDim.x < S ? a.W[e0 + q * blockDim.x] : 0;
#pragma unroll
        for (int q = 0; q < 4; q++)
            if (e0 + q * (int)blockDim.x < S) W[e0 + q * blockDim.x] = m61::lmul(v[q], ek);
    }
    __syncthreads();
    int off = 0;
    for (int c = 0; c < B; c++) {
        const int h = S >> (c + 1), n = h < NI ? h : NI;
        if (!zw) {
            const uint64_t z = za[c];
            uint64_t acc[5] = {0, 0, 0, 0, 0};
            for (int u = lt; u < h; u += NI) {
                const uint64_t w = W[h + u], b0 = Tb[u], b1 = Tb[u + h];
                range_pair(w, b0, b1, acc);
                fold_all<5>(acc);
                Tb[u] = fold(b0, b1, z);
            }
            if (lt < n)
#pragma unroll
                for (int q = 0; q < 5; q++) pr[(off + lt) * 5 + q] = acc[q];
        } else {
            const uint64_t z = zz[c];
            uint64_t acc[3] = {0, 0, 0};
            for (int u = lt; u < h; u += NI) {
                const uint64_t w = W[h + u];
                const uint64_t d0 = Td[u], d1 = Td[u + h], s0 = Ts[u], s1 = Ts[u + h];
                relu_pair(w, d0, d1, s0, s1, acc);
                fold_all<3>(acc);
                Td[u] = fold(d0, d1, z);
                Ts[u] = fold(s0, s1, z);
            }
            if (lt < n)
#pragma unroll
                for (int q = 0; q < 3; q++) pz[(off + lt) * 3 + q] = acc[q];
        }
        off += n;
        __syncthreads();
    }
    // per-round sums: sum q = 8 c + w over the round's thread entries (folded
    // values), eight lanes per sum, four terms added before each fold
    const int ntask = 64 * B;
    for (int task = tid; task < ntask; task += blockDim.x) {  // ntask is a multiple of 64: whole waves iterate
        const int q = task >> 3, part = task & 7, c = q >> 3, w = q & 7;
        int o = 0;
        for (int cc = 0; cc < c; cc++) o += (S >> (cc + 1)) < NI ? (S >> (cc + 1)) : NI;
        const int n = (S >> (c + 1)) < NI ? (S >> (c + 1)) : NI;
        const uint64_t *src = w < 5 ? pr + (size_t)o * 5 + w : pz + (size_t)o * 3 + (w - 5);
        const int st = w < 5 ? 5 : 3;
        uint64_t v = 0;
        if (w < 5 || RELU) {
            int e = part;
            for (; e + 24 < n; e += 32) v = m61::fold(v + src[e * st] + src[(e + 8) * st] + src[(e + 16) * st] + src[(e + 24) * st]);
            for (; e < n; e += 8) v = m61::fold(v + src[e * st]);
        }
        v = m61::fold(v + __shfl_xor(v, 1, 64));
        v = m61::fold(v + __shfl_xor(v, 2, 64));
        v = m61::fold(v + __shfl_xor(v, 4, 64));
        if (part == 0) red[q] = m61::canon(v);
    }
    __syncthreads();
    if (nsub > 1) {
        if (tid < 8 * B) a.part[(size_t)(tid >> 3) * a.stride + 8 * k + (tid & 7)] = red[tid];
        if (tid == 0) a.bx[k] = m61::canon(Tb[0]);
        if (RELU && tid == NI) {
            a.d[k] = m61::canon(Td[0]);
            a.s[k] = m61::canon(Ts[0]);
        }
    } else {
        // round c's evaluation X of instance zr by thread 8 c + 4 zr + X
        if (tid < 8 * B) {
            const int c = tid >> 3, zr = (tid >> 2) & 1, X = tid & 3;
            if (!zr || RELU)
                a.tr[(zr ? a.out2 : a.out0) + 4 * c + X] = x_round_eval(red + 8 * c, a.j + c, X, zr != 0, a.xc);
        }
        if (tid == 0) {
            *a.fin_b = m61::canon(Tb[0]);
            if (RELU) {
                const uint64_t inv2 = 1ull << 60;  // (p + 1) / 2
                const uint64_t d = m61::canon(Td[0]), sv = m61::canon(Ts[0]);
                *a.fin_r = m61::mul(m61::add(d, sv), inv2);
                *a.fin_y = m61::mul(m61::sub(sv, d), inv2);
            }
        }
    }
}

void launch_xblock(bool relu, bool first, const XBlockArgs &a, const XJobs &jobs, hipStream_t st)
{
    const int nmain = 1 << (a.lS - a.B);
    const dim3 g(nmain + jobs.nslot + jobs.nplane), b(kThreads);
    if (relu) hipLaunchKernelGGL(k_xblock<true>, g, b, 0, st, a, (int)first, jobs, nmain);
    else hipLaunchKernelGGL(k_xblock<false>, g, b, 0, st, a, (int)first, jobs, nmain);
}

}  // namespace ra
