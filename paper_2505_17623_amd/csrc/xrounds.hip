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
#include "gram_reduce.hpp"
#include "rsetup.hpp"
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

// Workgroups below nmain run the rounds; the others are jobs, then (first
// register pass of a range call) the range riders: the Gram reduction, the
// constant block and a deferred witness step, in the rounds' LDS.
template <int C, bool FIRST, bool RELU>
__global__ __launch_bounds__(256) void k_xrounds(XArgs a, uint64_t sub, int stride, XJobs jobs, int nmain,
                                                 RangeRiders rr)
{
    constexpr int NPB = RELU ? 128 : 256, NVR = 5 * C;
    __shared__ uint64_t smem[xrounds_lds_words<C>()];
    static_assert(xrounds_lds_words<C>() >= kGramReduceLdsWords && xrounds_lds_words<C>() >= kConstsLdsWords &&
                      xrounds_lds_words<C>() >= kClaimsLdsWords,
                  "the riders work in the rounds' LDS");
    if ((int)blockIdx.x >= nmain) {  // workgroup-uniform
        const int q = blockIdx.x - nmain, nj = jobs.nslot + jobs.nplane;
        if (q < nj) x_job(jobs, q, smem);
        else if (q - nj < rr.nred) gram_reduce_block(rr.gpart, rr.nblk, rr.tiles, rr.gsum, q - nj, smem);
        else if (q - nj == rr.nred) range_consts_block(rr.rc, smem);
        else witness_claims_block(rr.rc, smem);
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

int range_riders(const RangeRiders &r) { return r.nred + 1 + (r.rc.cj.nblk > 0 ? 1 : 0); }

void launch_xrounds(int C, bool first, bool relu, const XArgs &a, uint64_t S, int stride, const XJobs &jobs,
                    hipStream_t st, const RangeRiders *riders)
{
    const uint64_t sub = S >> C;
    const int nmain = xround_blocks(sub, relu);
    const RangeRiders none{};
    const RangeRiders &rr = riders ? *riders : none;
    const dim3 g(nmain + jobs.nslot + jobs.nplane + (riders ? range_riders(rr) : 0)), b(kThreads);
#define RA_X(CC, F, Z) hipLaunchKernelGGL((k_xrounds<CC, F, Z>), g, b, 0, st, a, sub, stride, jobs, nmain, rr)
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
// B rounds per sub-cube, one wave per sub-cube and instance.  Sub-cube k
// holds the 2^B entries k + u 2^(lS - B) (u < 2^B) of each table; entry u
// lives in lane u mod 64, slot u / 64 of the wave.  Round c pairs u and
// u + h (h = 2^(B-1-c)) with weight
//   eq(r_{j+c+1 .. j+B-1}, u) eq(r_{j+B ..}, k) = W[h + u] e_k,
// W the heap of suffix eq tables of the window r_{j+1 .. j+B-1} (set-up: the
// WS heap, or for the last pass the LS heap), e_k from the suffix heaps.
// While h >= 64 both entries of a pair sit in the same lane, so those rounds
// run in registers; the later ones take the partner from lane u + h by a
// cross-lane read.  No workgroup barrier is needed after the weights are
// staged.  The sums of a round are formed with the weights W alone and
// multiplied by e_k once, after the wave's lanes are summed (through a
// wave-private LDS area).  A pass over several sub-cubes writes one partial
// per round and sub-cube; the last pass (one sub-cube) writes the round
// polynomials and the final values.
// Workgroups take two sub-cubes with ReLU (waves 2i, 2i + 1: the range and
// the ReLU instance of sub-cube 2 blk + i), else four (one wave each).
// ---------------------------------------------------------------------------
constexpr int kXbMax = 1 << kXBlockMax;
constexpr int kXbRedStride = 65;                                   // LDS words per summed value (64 lanes + pad)
constexpr int kXbRedWords = 5 * kXBlockMax * kXbRedStride + 8 * kXBlockMax;  // per wave
constexpr int kXbLdsWords = kXbMax + 4 * kXbRedWords;
static_assert(kXbLdsWords >= kJobLdsWords, "jobs share the workgroup's LDS");

// Value of lane (lane + h) of the wave (h < 64; lanes past the end read
// their own value, unused).
__device__ __forceinline__ uint64_t lane_down(uint64_t v, int h) { return __shfl_down(v, (unsigned)h, 64); }

// The sub-cube of one wave: range t0 = Bx; ReLU t0 = D, t1 = S (from R, Y in
// the first pass); all loads issued at once.
template <int B, bool ZW>
__device__ __forceinline__ void xb_load(const XBlockArgs &a, bool first, uint64_t k, uint64_t nsub,
                                        uint64_t (&t0)[(1 << B) >= 64 ? (1 << B) / 64 : 1],
                                        uint64_t (&t1)[(1 << B) >= 64 ? (1 << B) / 64 : 1])
{
    constexpr int S = 1 << B, E = S >= 64 ? S / 64 : 1;
    const int lane = threadIdx.x & 63;
    if (!ZW) {
#pragma unroll
        for (int e = 0; e < E; e++) {
            const int u = e * 64 + lane;
            t0[e] = u < S ? a.bx[k + (uint64_t)u * nsub] : 0;
            t1[e] = 0;
        }
    } else if (first) {
        int32_t vr[E], vy[E];
#pragma unroll
        for (int e = 0; e < E; e++) {
            const int u = e * 64 + lane;
            vr[e] = u < S ? a.R[k + (uint64_t)u * nsub] : 0;
            vy[e] = u < S ? a.Y[k + (uint64_t)u * nsub] : 0;
        }
#pragma unroll
        for (int e = 0; e < E; e++) {
            t0[e] = small_to_field((int64_t)vr[e] - vy[e]);
            t1[e] = small_to_field((int64_t)vr[e] + vy[e]);
        }
    } else {
#pragma unroll
        for (int e = 0; e < E; e++) {
            const int u = e * 64 + lane;
            t0[e] = u < S ? a.d[k + (uint64_t)u * nsub] : 0;
            t1[e] = u < S ? a.s[k + (uint64_t)u * nsub] : 0;
        }
    }
}

// The B rounds of one wave over its sub-cube (t0, t1 from xb_load; W staged).
template <int B, bool ZW, bool RELU>
__device__ __forceinline__ void xb_wave(const XBlockArgs &a, uint64_t k, uint64_t nsub, const uint64_t *__restrict__ W,
                                        uint64_t *red, uint64_t ek, uint64_t (&t0)[(1 << B) >= 64 ? (1 << B) / 64 : 1],
                                        uint64_t (&t1)[(1 << B) >= 64 ? (1 << B) / 64 : 1])
{
    constexpr int S = 1 << B, NV = ZW ? 3 : 5, E = S >= 64 ? S / 64 : 1, NR = B > 0 ? B : 1;
    const int lane = threadIdx.x & 63;
    const uint64_t *rho = ZW ? a.rho_z : a.rho_a;
    uint64_t z[NR];
#pragma unroll
    for (int c = 0; c < B; c++) z[c] = rho[c];
    // the last pass: the constants of the evaluation this lane makes (round
    // lane / 4), fetched before the rounds
    static_assert(4 * kXTailLog <= 64, "one evaluation per lane in the last pass");
    XEvalK kc{};
    if (nsub == 1 && lane < 4 * B) kc = x_eval_consts(a.xc, a.j + (lane >> 2), ZW);
    // round c's sums of this lane go to red[(c NV + q) kXbRedStride + lane]
#pragma unroll
    for (int c = 0; c < B; c++) {
        const int h = S >> (c + 1);
        uint64_t acc[NV];
#pragma unroll
        for (int q = 0; q < NV; q++) acc[q] = 0;
        if (h >= 64) {  // both entries of every pair in this lane: slots e and e + h / 64
            const int hs = h / 64;
#pragma unroll
            for (int e = 0; e < E / 2; e++) {
                if (e < hs) {
                    const uint64_t w = W[h + e * 64 + lane];
                    if (!ZW) {
                        range_pair(w, t0[e], t0[e + hs], acc);
                        t0[e] = fold(t0[e], t0[e + hs], z[c]);
                    } else {
                        relu_pair(w, t0[e], t0[e + hs], t1[e], t1[e + hs], acc);
                        t0[e] = fold(t0[e], t0[e + hs], z[c]);
                        t1[e] = fold(t1[e], t1[e + hs], z[c]);
                    }
                    fold_all<NV>(acc);
                }
            }
        } else {  // lane u < h pairs with lane u + h (slot 0)
            const uint64_t p0 = lane_down(t0[0], h), p1 = ZW ? lane_down(t1[0], h) : 0;
            if (lane < h) {
                const uint64_t w = W[h + lane];
                if (!ZW) {
                    range_pair(w, t0[0], p0, acc);
                    t0[0] = fold(t0[0], p0, z[c]);
                } else {
                    relu_pair(w, t0[0], p0, t1[0], p1, acc);
                    t0[0] = fold(t0[0], p0, z[c]);
                    t1[0] = fold(t1[0], p1, z[c]);
                }
                fold_all<NV>(acc);
            }
        }
#pragma unroll
        for (int q = 0; q < NV; q++) red[(c * NV + q) * kXbRedStride + lane] = acc[q];
    }
    // lane sums of every (round, value) through the wave's LDS area: lane v
    // sums value v over the 64 lanes, four terms before each fold
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    uint64_t *tot = red + 5 * kXBlockMax * kXbRedStride;  // 8 words per round: the sums at e_k
    static_assert(kXBlockMax * 5 <= 64, "one lane per summed value");
    if (lane < B * NV) {
        const uint64_t *src = red + lane * kXbRedStride;
        uint64_t v0 = 0, v1 = 0;
#pragma unroll
        for (int l = 0; l < 64; l += 8) {
            v0 = m61::fold(v0 + src[l] + src[l + 1] + src[l + 2] + src[l + 3]);
            v1 = m61::fold(v1 + src[l + 4] + src[l + 5] + src[l + 6] + src[l + 7]);
        }
        const int c = lane / NV, q = lane % NV;
        tot[8 * c + (ZW ? 5 : 0) + q] = m61::canon(m61::lmul(m61::fold(v0 + v1), ek));
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (nsub > 1) {
        // round c's partial of sub-cube k: words 0-4 range, 5-7 ReLU (zero without it)
        for (int t = lane; t < 8 * B; t += 64) {  // 8 B may exceed the wave
            const int c = t >> 3, w = t & 7;
            const bool mine = ZW ? w >= 5 : w < 5;
            if (mine) a.part[(size_t)c * a.stride + 8 * k + w] = tot[t];
            else if (!RELU) a.part[(size_t)c * a.stride + 8 * k + w] = 0;
        }
        if (lane == 0) {
            if (!ZW) a.bx[k] = m61::canon(t0[0]);
            else {
                a.d[k] = m61::canon(t0[0]);
                a.s[k] = m61::canon(t1[0]);
            }
        }
    } else {
        // round c's evaluation X by lane 4 c + X
        for (int t = lane; t < 4 * B; t += 64) {
            const int c = t >> 2, X = t & 3;
            const int out = ZW ? a.out2 : a.out0;
            if (out >= 0) a.tr[out + 4 * c + X] = x_round_eval(tot + 8 * c, kc, X, ZW);
        }
        if (lane == 0) {
            if (!ZW) {
                *a.fin_b = m61::canon(t0[0]);
            } else {
                const uint64_t inv2 = 1ull << 60;  // (p + 1) / 2
                const uint64_t d = m61::canon(t0[0]), sv = m61::canon(t1[0]);
                *a.fin_r = m61::mul(m61::add(d, sv), inv2);
                *a.fin_y = m61::mul(m61::sub(sv, d), inv2);
            }
        }
    }
}

template <bool RELU, int B>
__global__ __launch_bounds__(256) void k_xblock(XBlockArgs a, int first, XJobs jobs, int nmain)
{
    __shared__ uint64_t smem[kXbLdsWords];
    if ((int)blockIdx.x >= nmain) {
        x_job(jobs, blockIdx.x - nmain, smem);
        return;
    }
    constexpr int S = 1 << B, PER = RELU ? 2 : 4, E = S >= 64 ? S / 64 : 1;  // sub-cubes per workgroup
    const int tid = threadIdx.x, wv = tid >> 6;
    const uint64_t nsub = 1ull << (a.lS - B);
    const uint64_t k = (uint64_t)blockIdx.x * PER + (RELU ? (wv >> 1) : wv);
    const bool live = k < nsub, zw = RELU && (wv & 1);  // wave-uniform
    // the wave's sub-cube and weight e_k are fetched while the window
    // weights are staged: the two global latencies overlap
    uint64_t t0[E], t1[E], ek = 0;
    if (live) {
        if (zw) xb_load<B, true>(a, first != 0, k, nsub, t0, t1);
        else xb_load<B, false>(a, first != 0, k, nsub, t0, t1);
        ek = suffix_weight(a.HS, a.LS, a.lN - a.j - B, a.L, k);
    }
    uint64_t *W = smem;  // W[1 .. S), shared by the workgroup's sub-cubes
    for (int e = tid + 1; e < S; e += 256) W[e] = a.W[e];
    __syncthreads();
    if (!live) return;  // after the only barrier
    uint64_t *red = smem + kXbMax + wv * kXbRedWords;
    if (zw) xb_wave<B, true, RELU>(a, k, nsub, W, red, ek, t0, t1);
    else xb_wave<B, false, RELU>(a, k, nsub, W, red, ek, t0, t1);
}

void launch_xblock(bool relu, bool first, const XBlockArgs &a, const XJobs &jobs, hipStream_t st)
{
    const int per = relu ? 2 : 4;
    const uint64_t nsub = 1ull << (a.lS - a.B);
    const int nmain = (int)((nsub + per - 1) / per);
    const dim3 g(nmain + jobs.nslot + jobs.nplane), b(kThreads);
#define RA_XB(BB)                                                                                 \
    case BB:                                                                                      \
        if (relu) hipLaunchKernelGGL((k_xblock<true, BB>), g, b, 0, st, a, (int)first, jobs, nmain);  \
        else hipLaunchKernelGGL((k_xblock<false, BB>), g, b, 0, st, a, (int)first, jobs, nmain);      \
        break;
    switch (a.B) {
        RA_XB(0) RA_XB(1) RA_XB(2) RA_XB(3) RA_XB(4) RA_XB(5) RA_XB(6) RA_XB(7) RA_XB(8) RA_XB(9)
        default: RA_XB(10)
    }
#undef RA_XB
}

}  // namespace ra
