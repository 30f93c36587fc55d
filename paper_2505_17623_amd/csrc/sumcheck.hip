// sumcheck.hip -- the prover's sum-check rounds (Sec. II-D) of the matrix
// product instance sum_l a(l) b(l) (degree 2, Eq. (4)), the constants of the
// concatenated range check, and the transcript assembly.  The rounds over x
// of the range and ReLU instances are in xrounds.hip.
//
// Variables are bound most-significant first, so round j pairs entry i with
// entry i + h of the current table (h = half its size): both halves stream
// contiguously.  The challenges are known before the first round (the
// verifier's coins are a given stream), so every round is launched back to
// back; a round writes per-block partial sums that one assembly kernel
// reduces at the end, and folds the tables in place: T[i] <- T[i] +
// rho (T[i + h] - T[i]) for i < h (thread i alone reads i and i + h).
#include "common.hpp"
#include "m61.hpp"
#include "assemble.hpp"
#include "plane_round.hpp"
#include "xsetup.hpp"

namespace ra {

template <int KIND> struct KindTraits;
template <> struct KindTraits<KIND_MATMUL> { static constexpr int NT = 2, D = 2; };

// Contribution of one pair (lo = T[i], hi = T[i + h]) to g(X), X = 0..D.
template <int KIND>
__device__ __forceinline__ void pair_contrib(const uint64_t (&lo)[3], const uint64_t (&hi)[3], uint64_t (&acc)[4])
{
    constexpr int NT = KindTraits<KIND>::NT, D = KindTraits<KIND>::D;
    uint64_t val[NT], dif[NT];
#pragma unroll
    for (int q = 0; q < NT; q++) {
        val[q] = lo[q];
        dif[q] = m61::sub(hi[q], lo[q]);
    }
#pragma unroll
    for (int X = 0; X <= D; X++) {
        acc[X] = m61::add(acc[X], m61::mul(val[0], val[1]));
        if (X < D)
#pragma unroll
            for (int q = 0; q < NT; q++) val[q] = m61::add(val[q], dif[q]);  // table value at X + 1
    }
}

// ---------------------------------------------------------------------------
// C consecutive rounds over tables in global memory, fused.  With S the
// current table size and S' = S / 2^C, thread i loads the 2^C entries
// i + t S' (t < 2^C) of every table -- the sub-cube of the C variables about
// to be bound -- and runs the C rounds on them in registers: round r pairs
// local entries (u, u + 2^(C-1-r)), which are exactly the global pairs of
// that round.  It then writes the bound value to T[i] (i < S'; no other
// thread reads below S').  Partials of round r go to part + r * stride.
// ---------------------------------------------------------------------------
template <int KIND, int C>
__device__ __forceinline__ void rounds_body(const InstArgs &in, uint64_t sub, int blk, int nblk, int stride,
                                            uint64_t *red)
{
    constexpr int NT = KindTraits<KIND>::NT, D = KindTraits<KIND>::D, L = 1 << C;
    uint64_t r[C];
#pragma unroll
    for (int c = 0; c < C; c++) r[c] = in.rho[c];
    uint64_t *T[3] = {in.t0, in.t1, in.t2};
    uint64_t acc[C * 4];
#pragma unroll
    for (int i = 0; i < C * 4; i++) acc[i] = 0;
    for (uint64_t i = (uint64_t)blk * blockDim.x + threadIdx.x; i < sub; i += (uint64_t)nblk * blockDim.x) {
        uint64_t v[3][L];
#pragma unroll
        for (int q = 0; q < NT; q++)
#pragma unroll
            for (int t = 0; t < L; t++) v[q][t] = T[q][i + t * sub];
#pragma unroll
        for (int c = 0; c < C; c++) {
            const int h = L >> (c + 1);
            uint64_t a4[4] = {0, 0, 0, 0};
#pragma unroll
            for (int u = 0; u < h; u++) {
                uint64_t lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0};
#pragma unroll
                for (int q = 0; q < NT; q++) {
                    lo[q] = v[q][u];
                    hi[q] = v[q][u + h];
                }
                pair_contrib<KIND>(lo, hi, a4);
#pragma unroll
                for (int q = 0; q < NT; q++) v[q][u] = m61::add(lo[q], m61::mul(r[c], m61::sub(hi[q], lo[q])));
            }
#pragma unroll
            for (int X = 0; X <= D; X++) acc[4 * c + X] = m61::add(acc[4 * c + X], a4[X]);
        }
#pragma unroll
        for (int q = 0; q < NT; q++) T[q][i] = v[q][0];
    }
    m61::block_sum<C * 4>(acc, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int c = 0; c < C; c++)
#pragma unroll
            for (int X = 0; X <= D; X++) in.part[(size_t)c * stride + (size_t)blk * (D + 1) + X] = acc[4 * c + X];
}

// ---------------------------------------------------------------------------
// C consecutive rounds over tables in global memory, fused.  With S the
// current table size and S' = S / 2^C, thread i loads the 2^C entries
// i + t S' (t < 2^C) of every table -- the sub-cube of the C variables about
// to be bound -- and runs the C rounds on them in registers: round r pairs
// local entries (u, u + 2^(C-1-r)), which are exactly the global pairs of
// that round.  It then writes the bound value to T[i] (i < S'; no other
// thread reads below S').  Partials of round r go to part + r * stride.
// ---------------------------------------------------------------------------
template <int KIND, int C>
__global__ __launch_bounds__(256) void k_rounds(InstArgs a, uint64_t sub, int stride)
{
    __shared__ uint64_t red[m61::block_sum_words(C * 4, kThreads)];
    rounds_body<KIND, C>(a, sub, blockIdx.x, gridDim.x, stride, red);
}

int round_blocks(uint64_t h)
{
    const uint64_t b = (h + kThreads - 1) / kThreads;
    return (int)(b < (uint64_t)kMaxBlocks ? (b ? b : 1) : (uint64_t)kMaxBlocks);
}

int fused_rounds_max(int) { return 2; }

void launch_rounds(int kind, int C, uint64_t *t0, uint64_t *t1, uint64_t *t2, uint64_t S, const uint64_t *rho,
                   const uint64_t *kp, uint64_t *part, int stride, hipStream_t st)
{
    const uint64_t sub = S >> C;
    const int nb = round_blocks(sub);
    const InstArgs a{t0, t1, t2, rho, kp, part};
#define RA_ROUNDS(K, CC) hipLaunchKernelGGL((k_rounds<K, CC>), dim3(nb), dim3(kThreads), 0, st, a, sub, stride)
#define RA_ROUNDS_K(K)               \
    switch (C) {                     \
    case 1: RA_ROUNDS(K, 1); break;  \
    case 2: RA_ROUNDS(K, 2); break;  \
    case 3: RA_ROUNDS(K, 3); break;  \
    default: RA_ROUNDS(K, 4); break; \
    }
    (void)kind;
    RA_ROUNDS_K(KIND_MATMUL)
#undef RA_ROUNDS_K
#undef RA_ROUNDS
}

// ---------------------------------------------------------------------------
// All remaining rounds in one workgroup once the tables fit in LDS.  Thread
// t (< min(h, blockDim)) of round j writes its D + 1 partial evaluations to
// part + j * stride + (D + 1) t; the assembly reduces them.  Also writes the
// tables' final values and, with no rounds at all, the sum a b.
// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(kTailThreads) void k_tail(TailArgs in)
{
    constexpr int NT = KindTraits<KIND>::NT, D = KindTraits<KIND>::D;
    __shared__ uint64_t sm[NT][kTailMax];
    __shared__ uint64_t rc[kTailMaxLog];  // the rounds' challenges, read once
    const int tid = threadIdx.x, v = in.v;
    const uint32_t S = 1u << v;
    const uint64_t *G[3] = {in.t0, in.t1, in.t2};
    if (tid < v) rc[tid] = in.rho[tid];
    for (uint32_t i = tid; i < S; i += blockDim.x)
#pragma unroll
        for (int q = 0; q < NT; q++) sm[q][i] = G[q][i];
    __syncthreads();
    if (v == 0 && in.sum_out && tid == 0) *in.sum_out = m61::mul(sm[0][0], sm[1][0]);  // no rounds: the sum is a b
    for (int j = 0; j < v; j++) {
        const uint32_t h = S >> (j + 1);
        const uint64_t r = rc[j];
        uint64_t acc[4] = {0, 0, 0, 0};
        for (uint32_t i = tid; i < h; i += blockDim.x) {
            uint64_t lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0};
#pragma unroll
            for (int q = 0; q < NT; q++) {
                lo[q] = sm[q][i];
                hi[q] = sm[q][i + h];
            }
            pair_contrib<KIND>(lo, hi, acc);
#pragma unroll
            for (int q = 0; q < NT; q++) sm[q][i] = m61::add(lo[q], m61::mul(r, m61::sub(hi[q], lo[q])));
        }
        if ((uint32_t)tid < h)
#pragma unroll
            for (int X = 0; X <= D; X++) in.part[(size_t)j * in.stride + (size_t)(D + 1) * tid + X] = acc[X];
        __syncthreads();  // folds of round j visible to round j + 1
    }
    if (tid == 0) {
        if (in.fin0) *in.fin0 = sm[0][0];
        if (in.fin1) *in.fin1 = sm[1][0];
        if (NT > 2 && in.fin2) *in.fin2 = sm[NT - 1][0];
    }
}

size_t tail_capacity(int) { return kTailMax; }
int tail_units(uint32_t h) { return (int)(h < (uint32_t)kTailThreads ? h : kTailThreads); }

void launch_tail(int kind, const TailArgs &a, hipStream_t st)
{
    (void)kind;
    hipLaunchKernelGGL(k_tail<KIND_MATMUL>, dim3(1), dim3(kTailThreads), 0, st, a);
}

// ---------------------------------------------------------------------------
// Concatenated range check: constants of the plane rounds.
//
// Over b(q, x) (q = plane, first log P variables) the summand is
//   eq(tau_p, q) EQ(x) b (b - 1) + mu W(q) EQ(x) b,   EQ(x) = eq((r1, r2), x),
// W(q) = lambda_g 2^bit.  While plane variable j is free (x still Boolean):
//   g_j(X) = K_j eq(tau_j, X) A_j(X) + mu Bw_j(X),
//   A_j(X)  = sum_x EQ(x) sum_p' eq(tau_{>j}, p') b_X (b_X - 1),
//   Bw_j(X) = sum_x EQ(x) sum_p' W_j(X, p') b_X,
// where K_j = eq(tau_{<j}, sigma_{<j}), W_j is W bound at sigma_{<j}, and
// b_X = b(sigma_{<j}, X, p', x).  A_j and Bw_j are quadratic in X, so the
// plane kernel sums them at X = 0, 1, 2 and the assembly extends to X = 3.
// After all plane rounds the summand is EQ(x) (Ep b^2 + (mu Wp - Ep) b) with
// Ep = eq(tau_p, sigma_p), Wp = W~(sigma_p), the rounds over x of xrounds.hip.
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int off_half(int P, int j) { return P - (P >> (j - 1)); }      // e_j, w2_j
__host__ __device__ constexpr int off_full(int P, int j) { return 2 * P - 2 * (P >> (j - 1)); }  // W_j

size_t range_consts_words(int) { return C_WORDS; }

__device__ __forceinline__ uint64_t eq1(uint64_t a, uint64_t b)
{
    return m61::add(m61::mul(a, b), m61::mul(m61::sub(1, a), m61::sub(1, b)));
}

// Block 0 (256 threads): the constant block; chal points at lambda1:
// lambda1..3, mu, tau_p (lP), sigma (lP + ...).  Further blocks: the set-up of
// the rounds over x.  Every operand is first staged in LDS.
__global__ __launch_bounds__(256) void k_range_setup(const uint64_t *__restrict__ chal,
                                                     const WitParams *__restrict__ prm,
                                                     const uint64_t *__restrict__ claims, int lP,
                                                     uint64_t *__restrict__ cst, uint64_t *__restrict__ range_sum,
                                                     uint64_t *__restrict__ lut, XSetupArgs xs)
{
    const int tid = threadIdx.x;
    if (blockIdx.x > 0) {  // the set-up of the rounds over x
        __shared__ uint64_t rl[64], sl[64], zl[64];
        if (tid < xs.lN) {
            rl[tid] = xs.r[tid];
            sl[tid] = xs.sigx[tid];
            zl[tid] = xs.rho2 ? xs.rho2[tid] : 0;
        }
        __syncthreads();
        x_setup_body(xs, (blockIdx.x - 1) * blockDim.x + tid, rl, sl, zl);
        return;
    }
    __shared__ uint64_t c[C_WORDS];
    __shared__ uint64_t eqs[64];
    __shared__ uint64_t ch[4 + 2 * kMaxPlaneLog], cl[3];
    __shared__ int pv[3];
    const int P = 1 << lP;
    if (tid < 4 + 2 * lP) ch[tid] = chal[tid];
    if (tid >= 64 && tid < 67) cl[tid - 64] = claims[tid - 64];
    if (tid == 128) {
        pv[0] = prm->s;
        pv[1] = prm->t;
        pv[2] = prm->relu;
    }
    for (int i = tid; i < C_WORDS; i += blockDim.x) c[i] = 0;
    __syncthreads();
    const int s = pv[0], t = pv[1], relu = pv[2];
    const uint64_t *lam = ch, mu = ch[3], *tau = ch + 4, *sig = ch + 4 + lP;
    // W_1 = W: plane q holds bit b of group g -> lambda_g 2^b
    for (int q = tid; q < P; q += blockDim.x) {
        int g = -1, b = 0;
        if (q < s) g = 0, b = q;
        else if (q < s + t + 2) g = 1, b = q - s;
        else if (relu && q < s + 2 * t + 4) g = 2, b = q - s - t - 2;
        c[C_W + q] = g < 0 ? 0 : m61::mul(lam[g], 1ull << b);
    }
    // e_j[p] = eq(tau_{j+1..lP}, p) for all rounds j at once
    for (int idx = tid; idx < P - 1; idx += blockDim.x) {
        int j = 1;
        while (idx >= off_half(P, j + 1)) j++;
        const int p = idx - off_half(P, j);
        uint64_t acc = 1;
        for (int i = 0; i < lP - j; i++) acc = m61::mul(acc, m61::eq1_bit(tau[j + i], (p >> (lP - j - 1 - i)) & 1));
        c[C_E + idx] = acc;
    }
    // eq(sigma_p, q) for every plane (for the byte tables below)
    for (int q = tid; q < 64; q += blockDim.x) {
        uint64_t a = 0;
        if (q < P) {
            a = 1;
            for (int i = 0; i < lP; i++) a = m61::mul(a, m61::eq1_bit(sig[i], (q >> (lP - 1 - i)) & 1));
        }
        eqs[q] = a;
    }
    __syncthreads();
    for (int j = 1; j <= lP; j++) {  // W_{j+1} = W_j bound at sigma_j; w2_j = 2 W_j[p + h] - W_j[p]
        const int h = P >> j;
        const uint64_t *Wj = c + C_W + off_full(P, j);
        for (int p = tid; p < h; p += blockDim.x) {
            c[C_W2 + off_half(P, j) + p] = m61::sub(m61::add(Wj[p + h], Wj[p + h]), Wj[p]);
            if (j < lP) c[C_W + off_full(P, j + 1) + p] = m61::add(Wj[p], m61::mul(sig[j - 1], m61::sub(Wj[p + h], Wj[p])));
        }
        __syncthreads();
    }
    if (tid == 0) {
        uint64_t K = 1;
        for (int j = 1; j <= lP; j++) {
            c[C_K + j - 1] = K;
            c[C_TAU + j - 1] = tau[j - 1];
            K = m61::mul(K, eq1(tau[j - 1], sig[j - 1]));
        }
        const uint64_t *Wl = c + C_W + off_full(P, lP);
        const uint64_t Wp = m61::add(Wl[0], m61::mul(sig[lP - 1], m61::sub(Wl[1], Wl[0])));
        c[C_EP] = K;                                           // Ep
        c[C_EP + 1] = m61::sub(m61::mul(mu, Wp), K);           // c = mu Wp - Ep
        c[C_EP + 2] = Wp;
        c[C_EP + 3] = mu;
        // claimed sum mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~); claims = (R~, Rm~, Y~, Z~)
        uint64_t H = m61::add(m61::mul(lam[0], cl[1]), m61::mul(lam[1], m61::add(cl[0], 1ull << (t + 1))));
        if (relu) H = m61::add(H, m61::mul(lam[2], cl[2]));
        *range_sum = m61::mul(mu, H);
    }
    __syncthreads();
    for (int i = tid; i < C_WORDS; i += blockDim.x) cst[i] = c[i];
    // lut[b][v] = sum over the set bits i of v of eq(sigma_p, 8 b + i)
    for (int i = tid; i < 8 * 256; i += blockDim.x) {
        const int b = i >> 8, v = i & 255;
        uint64_t a = 0;
        for (int k = 0; k < 8; k++)
            if ((v >> k) & 1) a += eqs[8 * b + k];
        lut[i] = m61::canon(a);
    }
}

void launch_range_setup(const uint64_t *chal, const WitParams *params, const uint64_t *claims, int lP, uint64_t *cst,
                        uint64_t *tr_range_sum, uint64_t *lut, const XSetupArgs &xs, hipStream_t st)
{
    const int xb = (x_setup_count(xs) + 255) / 256;
    hipLaunchKernelGGL(k_range_setup, dim3(1 + xb), dim3(256), 0, st, chal, params, claims, lP, cst, tr_range_sum,
                       lut, xs);
}

// ---------------------------------------------------------------------------
// Transcript assembly: reduce every slot's per-block partials and write the
// round evaluations (plane rounds combined as described above).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_assemble(SlotTable slots, const uint64_t *__restrict__ part, int part_stride,
                                                  uint64_t *__restrict__ tr, XConst xc, PlaneArgs pa)
{
    __shared__ uint64_t lds[kJobLdsWords];
    const int si = blockIdx.x;
    if (si >= slots.count) {  // a plane round
        plane_round(pa, si - slots.count + 1, lds);
        return;
    }
    assemble_slot(slots.s[si], part + (size_t)si * part_stride, tr, xc, lds);
}

void launch_assemble(const SlotTable &slots, const uint64_t *part, int part_stride, uint64_t *tr, const XConst &xc,
                     const PlaneArgs &pa, hipStream_t st)
{
    if (slots.count + pa.lP == 0) return;
    hipLaunchKernelGGL(k_assemble, dim3(slots.count + pa.lP), dim3(256), 0, st, slots, part, part_stride, tr, xc, pa);
}

}  // namespace ra

namespace ra {
// Kernel attributes set once per process (none needed at present).
void init_kernel_attributes() {}
}  // namespace ra
