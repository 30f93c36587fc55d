// sumcheck.hip -- the prover's sum-check rounds (Sec. II-D) for the three
// instances of a layer:
//   KIND_MATMUL  sum_l a(l) b(l)                              degree 2  (Eq. (4))
//   KIND_RANGE   sum_x EQ(x) (Ep b(x)^2 + c b(x))             degree 3  (range check,
//                after its plane variables are bound; Ep, c constants)
//   KIND_RELU    sum_x EQ(x) (R(x)^2 - Y(x)^2)                degree 3  (Eq. (6))
// and the fused kernel that binds the plane variables of the concatenated
// range check directly from the packed bit words.
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

namespace ra {

template <int KIND> struct KindTraits;
template <> struct KindTraits<KIND_MATMUL> { static constexpr int NT = 2, D = 2; };
template <> struct KindTraits<KIND_RANGE> { static constexpr int NT = 2, D = 3; };
template <> struct KindTraits<KIND_RELU> { static constexpr int NT = 3, D = 3; };

// Contribution of one pair (lo = T[i], hi = T[i + h]) to g(X), X = 0..D.
template <int KIND>
__device__ __forceinline__ void pair_contrib(const uint64_t (&lo)[3], const uint64_t (&hi)[3], uint64_t ep,
                                             uint64_t cc, uint64_t (&acc)[4])
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
        uint64_t f;
        if (KIND == KIND_MATMUL) {
            f = m61::mul(val[0], val[1]);
        } else if (KIND == KIND_RANGE) {
            f = m61::mul(val[0], m61::mul(val[1], m61::add(m61::mul(ep, val[1]), cc)));
        } else {
            f = m61::mul(val[0], m61::mul(m61::sub(val[1], val[2]), m61::add(val[1], val[2])));
        }
        acc[X] = m61::add(acc[X], f);
        if (X < D)
#pragma unroll
            for (int q = 0; q < NT; q++) val[q] = m61::add(val[q], dif[q]);  // table value at X + 1
    }
}

// ---------------------------------------------------------------------------
// One round over tables in global memory: evaluate, then fold in place.
// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(256) void k_round(uint64_t *__restrict__ t0, uint64_t *__restrict__ t1,
                                               uint64_t *__restrict__ t2, uint64_t h, const uint64_t *__restrict__ rho_p,
                                               const uint64_t *__restrict__ kp, uint64_t *__restrict__ part)
{
    constexpr int NT = KindTraits<KIND>::NT, D = KindTraits<KIND>::D;
    __shared__ uint64_t red[4 * 4];
    const uint64_t rho = *rho_p;
    const uint64_t ep = KIND == KIND_RANGE ? kp[0] : 0, cc = KIND == KIND_RANGE ? kp[1] : 0;
    uint64_t *T[3] = {t0, t1, t2};
    uint64_t acc[4] = {0, 0, 0, 0};
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < h; i += (uint64_t)gridDim.x * blockDim.x) {
        uint64_t lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0};
#pragma unroll
        for (int q = 0; q < NT; q++) {
            lo[q] = T[q][i];
            hi[q] = T[q][i + h];
        }
        pair_contrib<KIND>(lo, hi, ep, cc, acc);
#pragma unroll
        for (int q = 0; q < NT; q++) T[q][i] = m61::add(lo[q], m61::mul(rho, m61::sub(hi[q], lo[q])));
    }
    m61::block_sum<4>(acc, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int X = 0; X <= D; X++) part[(size_t)blockIdx.x * (D + 1) + X] = acc[X];
}

int round_blocks(uint64_t h)
{
    const uint64_t b = (h + kThreads - 1) / kThreads;
    return (int)(b < (uint64_t)kMaxBlocks ? (b ? b : 1) : (uint64_t)kMaxBlocks);
}

void launch_round(int kind, uint64_t *t0, uint64_t *t1, uint64_t *t2, uint64_t h, const uint64_t *rho,
                  const uint64_t *kp, uint64_t *part, hipStream_t st)
{
    const int nb = round_blocks(h);
    switch (kind) {
    case KIND_MATMUL: hipLaunchKernelGGL(k_round<KIND_MATMUL>, dim3(nb), dim3(kThreads), 0, st, t0, t1, t2, h, rho, kp, part); break;
    case KIND_RANGE: hipLaunchKernelGGL(k_round<KIND_RANGE>, dim3(nb), dim3(kThreads), 0, st, t0, t1, t2, h, rho, kp, part); break;
    default: hipLaunchKernelGGL(k_round<KIND_RELU>, dim3(nb), dim3(kThreads), 0, st, t0, t1, t2, h, rho, kp, part); break;
    }
}

// ---------------------------------------------------------------------------
// All remaining rounds in one workgroup once the tables fit in LDS.
// Writes the evaluations of every round, the tables' final values, and (if
// sum_out is set) the hypercube sum of the summand before the first round.
// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(1024) void k_tail(const uint64_t *__restrict__ t0, const uint64_t *__restrict__ t1,
                                               const uint64_t *__restrict__ t2, int v, const uint64_t *__restrict__ rho,
                                               const uint64_t *__restrict__ kp, uint64_t *__restrict__ evals,
                                               uint64_t *fin0, uint64_t *fin1, uint64_t *fin2, uint64_t *sum_out)
{
    constexpr int NT = KindTraits<KIND>::NT, D = KindTraits<KIND>::D;
    extern __shared__ uint64_t sm[];
    __shared__ uint64_t red[4 * 16];
    const uint32_t S = 1u << v;
    uint64_t *T[3] = {sm, sm + S, sm + 2 * S};
    const uint64_t *G[3] = {t0, t1, t2};
    for (uint32_t i = threadIdx.x; i < S; i += blockDim.x)
#pragma unroll
        for (int q = 0; q < NT; q++) T[q][i] = G[q][i];
    __syncthreads();
    const uint64_t ep = KIND == KIND_RANGE ? kp[0] : 0, cc = KIND == KIND_RANGE ? kp[1] : 0;

    if (sum_out) {  // sum over the hypercube of a(x) b(x) (matrix instance only)
        uint64_t acc[4] = {0, 0, 0, 0};
        for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) acc[0] = m61::add(acc[0], m61::mul(T[0][i], T[1][i]));
        m61::block_sum<4>(acc, red);
        if (threadIdx.x == 0) *sum_out = acc[0];
    }
    for (int j = 0; j < v; j++) {
        const uint32_t h = S >> (j + 1);
        const uint64_t r = rho[j];
        uint64_t acc[4] = {0, 0, 0, 0};
        for (uint32_t i = threadIdx.x; i < h; i += blockDim.x) {
            uint64_t lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0};
#pragma unroll
            for (int q = 0; q < NT; q++) {
                lo[q] = T[q][i];
                hi[q] = T[q][i + h];
            }
            pair_contrib<KIND>(lo, hi, ep, cc, acc);
#pragma unroll
            for (int q = 0; q < NT; q++) T[q][i] = m61::add(lo[q], m61::mul(r, m61::sub(hi[q], lo[q])));
        }
        m61::block_sum<4>(acc, red);  // ends with a barrier: folds are visible to the next round
        if (threadIdx.x == 0)
#pragma unroll
            for (int X = 0; X <= D; X++) evals[(size_t)j * (D + 1) + X] = acc[X];
    }
    if (threadIdx.x == 0) {
        if (fin0) *fin0 = T[0][0];
        if (fin1) *fin1 = T[1][0];
        if (NT > 2 && fin2) *fin2 = T[2][0];
    }
}

size_t tail_capacity(int ntab) { return kTailLdsBytes / (8 * (size_t)ntab) >= 8192 ? 8192 : 4096; }

void launch_tail(int kind, const uint64_t *t0, const uint64_t *t1, const uint64_t *t2, int v, const uint64_t *rho,
                 const uint64_t *kp, uint64_t *evals, uint64_t *finals, uint64_t *sum_out, hipStream_t st)
{
    // finals[0..NT) receive the tables' final values (a null entry is skipped)
    uint64_t *f0 = finals ? finals : nullptr, *f1 = finals ? finals + 1 : nullptr, *f2 = finals ? finals + 2 : nullptr;
    const int nt = kind == KIND_RELU ? 3 : 2;
    const size_t lds = (size_t)nt * 8 * ((size_t)1 << v);
    switch (kind) {
    case KIND_MATMUL: hipLaunchKernelGGL(k_tail<KIND_MATMUL>, dim3(1), dim3(kTailThreads), lds, st, t0, t1, t2, v, rho, kp, evals, f0, f1, f2, sum_out); break;
    case KIND_RANGE: hipLaunchKernelGGL(k_tail<KIND_RANGE>, dim3(1), dim3(kTailThreads), lds, st, t0, t1, t2, v, rho, kp, evals, f0, f1, f2, sum_out); break;
    default: hipLaunchKernelGGL(k_tail<KIND_RELU>, dim3(1), dim3(kTailThreads), lds, st, t0, t1, t2, v, rho, kp, evals, f0, f1, f2, sum_out); break;
    }
}

// Partial sums of a dot product (the matrix instance's claimed sum when its
// tables exceed the LDS tail).
__global__ __launch_bounds__(256) void k_dot(const uint64_t *__restrict__ a, const uint64_t *__restrict__ b,
                                             uint64_t len, uint64_t *__restrict__ part)
{
    __shared__ uint64_t red[4 * 4];
    uint64_t acc[4] = {0, 0, 0, 0};
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < len; i += (uint64_t)gridDim.x * blockDim.x)
        acc[0] = m61::add(acc[0], m61::mul(a[i], b[i]));
    m61::block_sum<4>(acc, red);
    if (threadIdx.x == 0) part[blockIdx.x] = acc[0];
}

void launch_dot(const uint64_t *a, const uint64_t *b, uint64_t len, uint64_t *part, hipStream_t st)
{
    hipLaunchKernelGGL(k_dot, dim3(round_blocks(len)), dim3(kThreads), 0, st, a, b, len, part);
}

__global__ __launch_bounds__(256) void k_i32_to_field(const int32_t *__restrict__ src, uint64_t N,
                                                      uint64_t *__restrict__ dst)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N; i += (uint64_t)gridDim.x * blockDim.x)
        dst[i] = m61::from_i64(src[i]);
}

void launch_i32_to_field(const int32_t *src, uint64_t N, uint64_t *dst, hipStream_t st)
{
    hipLaunchKernelGGL(k_i32_to_field, dim3(round_blocks(N)), dim3(kThreads), 0, st, src, N, dst);
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
// Ep = eq(tau_p, sigma_p), Wp = W~(sigma_p): the KIND_RANGE instance.
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int off_half(int P, int j) { return P - (P >> (j - 1)); }      // e_j, w2_j
__host__ __device__ constexpr int off_full(int P, int j) { return 2 * P - 2 * (P >> (j - 1)); }  // W_j

size_t range_consts_words(int) { return C_WORDS; }

__device__ __forceinline__ uint64_t eq1(uint64_t a, uint64_t b)
{
    return m61::add(m61::mul(a, b), m61::mul(m61::sub(1, a), m61::sub(1, b)));
}

// One thread.  chal points at lambda1: lambda1..3, mu, tau_p (lP), sigma (lP + ...).
__global__ void k_range_setup(const uint64_t *__restrict__ chal, const WitParams *__restrict__ prm,
                              const uint64_t *__restrict__ claims, int lP, uint64_t *__restrict__ cst,
                              uint64_t *__restrict__ range_sum)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const int P = 1 << lP;
    const int s = prm->s, t = prm->t, relu = prm->relu;
    const uint64_t *lam = chal, mu = chal[3], *tau = chal + 4, *sig = chal + 4 + lP;
    for (int i = 0; i < C_WORDS; i++) cst[i] = 0;
    // W_1 = W
    uint64_t *W1 = cst + C_W;
    int q = 0;
    for (int b = 0; b < s; b++, q++) W1[q] = m61::mul(lam[0], 1ull << b);
    for (int b = 0; b < t + 2; b++, q++) W1[q] = m61::mul(lam[1], 1ull << b);
    if (relu)
        for (int b = 0; b < t + 2; b++, q++) W1[q] = m61::mul(lam[2], 1ull << b);
    uint64_t K = 1;
    for (int j = 1; j <= lP; j++) {
        const int h = P >> j;  // pairs in round j
        uint64_t *e = cst + C_E + off_half(P, j);
        uint64_t *Wj = cst + C_W + off_full(P, j);
        uint64_t *w2 = cst + C_W2 + off_half(P, j);
        for (int p = 0; p < h; p++) {  // eq(tau_{j+1..lP}, p')
            uint64_t acc = 1;
            for (int i = 0; i < lP - j; i++) acc = m61::mul(acc, m61::eq1_bit(tau[j + i], (p >> (lP - j - 1 - i)) & 1));
            e[p] = acc;
            w2[p] = m61::sub(m61::add(Wj[p + h], Wj[p + h]), Wj[p]);
        }
        cst[C_K + j - 1] = K;
        cst[C_TAU + j - 1] = tau[j - 1];
        if (j < lP) {  // W_{j+1} = W_j bound at sigma_j
            uint64_t *Wn = cst + C_W + off_full(P, j + 1);
            for (int p = 0; p < h; p++) Wn[p] = m61::add(Wj[p], m61::mul(sig[j - 1], m61::sub(Wj[p + h], Wj[p])));
        }
        K = m61::mul(K, eq1(tau[j - 1], sig[j - 1]));
    }
    // fully bound: Wp = W_lP bound at sigma_lP
    const uint64_t *Wl = cst + C_W + off_full(P, lP);
    const uint64_t Wp = m61::add(Wl[0], m61::mul(sig[lP - 1], m61::sub(Wl[1], Wl[0])));
    cst[C_EP] = K;                                                  // Ep
    cst[C_EP + 1] = m61::sub(m61::mul(mu, Wp), K);                 // c = mu Wp - Ep
    cst[C_EP + 2] = Wp;
    cst[C_EP + 3] = mu;
    // claimed sum mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~); claims = (R~, Rm~, Y~, Z~)
    uint64_t H = m61::add(m61::mul(lam[0], claims[1]), m61::mul(lam[1], m61::add(claims[0], 1ull << (t + 1))));
    if (relu) H = m61::add(H, m61::mul(lam[2], claims[2]));
    *range_sum = m61::mul(mu, H);
}

void launch_range_setup(const uint64_t *chal, const WitParams *params, const uint64_t *claims, int lP, uint64_t *cst,
                        uint64_t *tr_range_sum, hipStream_t st)
{
    hipLaunchKernelGGL(k_range_setup, dim3(1), dim3(64), 0, st, chal, params, claims, lP, cst, tr_range_sum);
}

int plane_blocks(uint64_t N)
{
    const uint64_t b = (N + kThreads - 1) / kThreads;
    return (int)(b < (uint64_t)kMaxBlocks ? b : (uint64_t)kMaxBlocks);
}

// Plane rounds, one output x per thread: all lP rounds from the packed word.
// Partials of round j go to part + j * kMaxBlocks * 6 + block * 6.
template <int LP>
__global__ __launch_bounds__(256) void k_plane(const uint64_t *__restrict__ bits, uint64_t N, int lk,
                                               const uint64_t *__restrict__ E1, const uint64_t *__restrict__ E2,
                                               const uint64_t *__restrict__ cst, const uint64_t *__restrict__ sigma,
                                               uint64_t *__restrict__ EQ, uint64_t *__restrict__ EQ2,
                                               uint64_t *__restrict__ Bx, uint64_t *__restrict__ part)
{
    constexpr int P = 1 << LP;
    __shared__ uint64_t s_c[C_W2 + 64];
    __shared__ uint64_t s_sig[LP];
    __shared__ uint64_t red[6 * LP * 4];
    for (int i = threadIdx.x; i < C_W2 + 64; i += blockDim.x) s_c[i] = cst[i];
    if (threadIdx.x < LP) s_sig[threadIdx.x] = sigma[threadIdx.x];
    __syncthreads();
    const uint64_t kmask = (1ull << lk) - 1;
    uint64_t acc[LP * 6];
#pragma unroll
    for (int i = 0; i < LP * 6; i++) acc[i] = 0;

    for (uint64_t x = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; x < N; x += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t w = bits[x];
        const uint64_t eqx = m61::mul(E1[x >> lk], E2[x & kmask]);
        EQ[x] = eqx;
        if (EQ2) EQ2[x] = eqx;
        uint64_t v[P / 2];
        {   // round 1: the pair values are bits
            constexpr int h = P / 2;
            const uint64_t *e = s_c + C_E + off_half(P, 1);
            const uint64_t *W = s_c + C_W + off_full(P, 1);
            const uint64_t *w2 = s_c + C_W2 + off_half(P, 1);
            const uint64_t sg = s_sig[0], one_m = m61::sub(1, sg);
            uint64_t a2 = 0, b0 = 0, b1 = 0, b2 = 0;
#pragma unroll
            for (int i = 0; i < h; i++) {
                const uint32_t lo = (uint32_t)(w >> i) & 1u, hi = (uint32_t)(w >> (i + h)) & 1u;
                if (lo != hi) a2 = m61::add(a2, e[i]);  // (2hi - lo)(2hi - lo - 1) = 2
                if (lo) b0 = m61::add(b0, W[i]);
                if (hi) b1 = m61::add(b1, W[i + h]);
                if (hi) b2 = m61::add(b2, lo ? w2[i] : m61::add(w2[i], w2[i]));
                else if (lo) b2 = m61::sub(b2, w2[i]);
                v[i] = lo ? (hi ? 1 : one_m) : (hi ? sg : 0);
            }
            a2 = m61::add(a2, a2);
            acc[2] = m61::add(acc[2], m61::mul(eqx, a2));
            acc[3] = m61::add(acc[3], m61::mul(eqx, b0));
            acc[4] = m61::add(acc[4], m61::mul(eqx, b1));
            acc[5] = m61::add(acc[5], m61::mul(eqx, b2));
        }
#pragma unroll
        for (int j = 2; j <= LP; j++) {
            const int h = P >> j;
            const uint64_t *e = s_c + C_E + off_half(P, j);
            const uint64_t *W = s_c + C_W + off_full(P, j);
            const uint64_t *w2 = s_c + C_W2 + off_half(P, j);
            const uint64_t sg = s_sig[j - 1];
            uint64_t a0 = 0, a1 = 0, a2 = 0, b0 = 0, b1 = 0, b2 = 0;
#pragma unroll
            for (int i = 0; i < h; i++) {
                const uint64_t lo = v[i], hi = v[i + h];
                const uint64_t d = m61::sub(hi, lo), x2 = m61::add(hi, d);
                a0 = m61::add(a0, m61::mul(e[i], m61::mul(lo, m61::sub(lo, 1))));
                a1 = m61::add(a1, m61::mul(e[i], m61::mul(hi, m61::sub(hi, 1))));
                a2 = m61::add(a2, m61::mul(e[i], m61::mul(x2, m61::sub(x2, 1))));
                b0 = m61::add(b0, m61::mul(W[i], lo));
                b1 = m61::add(b1, m61::mul(W[i + h], hi));
                b2 = m61::add(b2, m61::mul(w2[i], x2));
                v[i] = m61::add(lo, m61::mul(sg, d));
            }
            uint64_t *ac = acc + 6 * (j - 1);
            ac[0] = m61::add(ac[0], m61::mul(eqx, a0));
            ac[1] = m61::add(ac[1], m61::mul(eqx, a1));
            ac[2] = m61::add(ac[2], m61::mul(eqx, a2));
            ac[3] = m61::add(ac[3], m61::mul(eqx, b0));
            ac[4] = m61::add(ac[4], m61::mul(eqx, b1));
            ac[5] = m61::add(ac[5], m61::mul(eqx, b2));
        }
        Bx[x] = v[0];
    }
    m61::block_sum<LP * 6>(acc, red);
    if (threadIdx.x == 0)
#pragma unroll
        for (int j = 0; j < LP; j++)
#pragma unroll
            for (int i = 0; i < 6; i++) part[(size_t)j * kMaxBlocks * 6 + (size_t)blockIdx.x * 6 + i] = acc[6 * j + i];
}

void launch_plane_rounds(int lP, const uint64_t *bits, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2,
                         const uint64_t *cst, const uint64_t *sigma, uint64_t *EQ, uint64_t *EQ2, uint64_t *Bx,
                         uint64_t *part, hipStream_t st)
{
    const int nb = plane_blocks(N);
#define RA_PLANE_CASE(L)                                                                                           \
    case L: hipLaunchKernelGGL(k_plane<L>, dim3(nb), dim3(kThreads), 0, st, bits, N, lk, E1, E2, cst, sigma, EQ, EQ2, Bx, part); break;
    switch (lP) {
        RA_PLANE_CASE(1)
        RA_PLANE_CASE(2)
        RA_PLANE_CASE(3)
        RA_PLANE_CASE(4)
        RA_PLANE_CASE(5)
        RA_PLANE_CASE(6)
    default: break;
    }
#undef RA_PLANE_CASE
}

// ---------------------------------------------------------------------------
// Transcript assembly: reduce every slot's per-block partials and write the
// round evaluations (plane rounds combined as described above).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_assemble(SlotTable slots, const uint64_t *__restrict__ part, int part_stride,
                                                  const uint64_t *__restrict__ cst, uint64_t *__restrict__ tr)
{
    __shared__ uint64_t red[6 * 4];
    for (int si = 0; si < slots.count; si++) {
        const Slot sl = slots.s[si];
        const uint64_t *p = part + (size_t)si * part_stride;
        uint64_t acc[6] = {0, 0, 0, 0, 0, 0};
        for (int b = threadIdx.x; b < sl.nblk; b += blockDim.x)
            for (int i = 0; i < sl.width; i++) acc[i] = m61::add(acc[i], p[(size_t)b * sl.width + i]);
        m61::block_sum<6>(acc, red);
        if (threadIdx.x == 0) {
            if (sl.kind == 1) {
                const int j = sl.round;  // 1-based plane round
                const uint64_t K = cst[C_K + j - 1], tau = cst[C_TAU + j - 1], mu = cst[C_EP + 3];
                // quadratic extension to X = 3: f(3) = f(0) - 3 f(1) + 3 f(2)
                uint64_t A[4] = {acc[0], acc[1], acc[2], 0}, B[4] = {acc[3], acc[4], acc[5], 0};
                A[3] = m61::add(A[0], m61::mul(3, m61::sub(A[2], A[1])));
                B[3] = m61::add(B[0], m61::mul(3, m61::sub(B[2], B[1])));
                for (int X = 0; X < 4; X++)
                    tr[sl.out + X] = m61::add(m61::mul(m61::mul(K, m61::eq1_small(tau, X)), A[X]), m61::mul(mu, B[X]));
            } else {
                for (int i = 0; i < sl.width; i++) tr[sl.out + i] = acc[i];
            }
        }
    }
}

void launch_assemble(const SlotTable &slots, const uint64_t *part, int part_stride, const uint64_t *cst, int lP,
                     uint64_t *tr, hipStream_t st)
{
    (void)lP;
    if (slots.count == 0) return;
    hipLaunchKernelGGL(k_assemble, dim3(1), dim3(256), 0, st, slots, part, part_stride, cst, tr);
}

}  // namespace ra

namespace ra {
// The LDS tail uses up to kTailLdsBytes of dynamic LDS.
void init_kernel_attributes()
{
    hipFuncSetAttribute((const void *)k_tail<KIND_MATMUL>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTailLdsBytes);
    hipFuncSetAttribute((const void *)k_tail<KIND_RANGE>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTailLdsBytes);
    hipFuncSetAttribute((const void *)k_tail<KIND_RELU>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTailLdsBytes);
}
}  // namespace ra
