// sumcheck.hip -- the prover's sum-check rounds (Sec. II-D) of the matrix
// product instance sum_l a(l) b(l) (degree 2, Eq. (4)) and the constants of
// the concatenated range check.  The rounds over x of the range and ReLU
// instances are in xrounds.hip.
//
// Variables are bound most-significant first, so round j pairs entry i with
// entry i + h of the current table (h = half its size): both halves stream
// contiguously.  The challenges are known before the first round (the
// verifier's coins are a given stream), so every round is launched back to
// back; the global rounds write per-block partial sums, and the LDS tail that
// finishes the instance also reduces them (extra workgroups) and its own
// rounds into the transcript.  Tables fold in place: T[i] <- T[i] +
// rho (T[i + h] - T[i]) for i < h (thread i alone reads i and i + h).
#include "common.hpp"
#include "m61.hpp"
#include "assemble.hpp"
#include "plane_round.hpp"

namespace ra {

template <int KIND> struct KindTraits;
template <> struct KindTraits<KIND_MATMUL> { static constexpr int NT = 2, D = 2; };

// Contribution of one pair (lo = T[i], hi = T[i + h]) to g(X), X = 0..D:
// acc[X] += a_X b_X with T_X = lo + X (hi - lo), added without folding (each
// term is a folded value; callers fold at least every fourth pair).
template <int KIND>
__device__ __forceinline__ void pair_contrib(const uint64_t (&lo)[3], const uint64_t (&hi)[3], uint64_t (&acc)[4])
{
    const uint64_t a2 = m61::lsub(2 * hi[0], lo[0]), b2 = m61::lsub(2 * hi[1], lo[1]);
    acc[0] += m61::lmul(lo[0], lo[1]);
    acc[1] += m61::lmul(hi[0], hi[1]);
    acc[2] += m61::lmul(a2, b2);
}

// lo + r (hi - lo), folded.
__device__ __forceinline__ uint64_t fold_to(uint64_t lo, uint64_t hi, uint64_t r)
{
    return m61::fold(lo + m61::lmul(r, m61::lsub(hi, lo)));
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
                for (int q = 0; q < NT; q++) v[q][u] = fold_to(lo[q], hi[q], r[c]);
                if ((u & 3) == 3 || u == h - 1)
#pragma unroll
                    for (int X = 0; X <= D; X++) a4[X] = m61::fold(a4[X]);
            }
#pragma unroll
            for (int X = 0; X <= D; X++) acc[4 * c + X] = m61::fold(acc[4 * c + X] + a4[X]);
        }
#pragma unroll
        for (int q = 0; q < NT; q++) T[q][i] = m61::canon(v[q][0]);
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
// All remaining rounds in one workgroup once the tables fit in LDS, and the
// assembly of the whole instance: workgroup 0 runs the rounds, keeps each
// thread's sums of a round in LDS, reduces them per round and writes the
// rounds' evaluations (and, for round 0, the claimed sum g(0) + g(1)); the
// further workgroups assemble the slots of the global rounds before it.
// Also writes the tables' final values and, with no rounds at all, the sum a b.
// ---------------------------------------------------------------------------
constexpr int kTailRounds = 767;  // sum over rounds of min(h, 256) for tables of <= 1024 entries
constexpr int kTailLdsWords = 2 * kTailMax + 3 * kTailRounds + 3 * kTailMaxLog + kTailMaxLog;
constexpr int kTailSmem = kTailLdsWords > kJobLdsWords ? kTailLdsWords : kJobLdsWords;

template <int KIND>
__global__ __launch_bounds__(kTailThreads) void k_tail(TailArgs in, XJobs jobs)
{
    constexpr int D = KindTraits<KIND>::D;
    __shared__ uint64_t smem[kTailSmem];
    if (blockIdx.x > 0) {
        const int q = blockIdx.x - 1;
        assemble_slot(jobs.s[q], jobs.part + (size_t)q * jobs.stride, jobs.tr, jobs.xc, smem);
        return;
    }
    uint64_t *ta = smem, *tb = ta + kTailMax, *pe = tb + kTailMax, *red = pe + 3 * kTailRounds, *rc = red + 3 * kTailMaxLog;
    const int tid = threadIdx.x, v = in.v, NI = blockDim.x;
    const int S = 1 << v;
    if (tid < v) rc[tid] = in.rho[tid];
    for (int i0 = tid; i0 < S; i0 += 4 * NI) {  // loads first
        uint64_t x[4], y[4];
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int i = i0 + q * NI;
            x[q] = i < S ? in.t0[i] : 0;
            y[q] = i < S ? in.t1[i] : 0;
        }
#pragma unroll
        for (int q = 0; q < 4; q++)
            if (i0 + q * NI < S) {
                ta[i0 + q * NI] = x[q];
                tb[i0 + q * NI] = y[q];
            }
    }
    __syncthreads();
    if (v == 0 && in.j0 == 0 && in.sum_out >= 0 && tid == 0)
        in.tr[in.sum_out] = m61::mul(ta[0], tb[0]);  // no rounds: the sum is a b
    int off = 0;
    for (int j = 0; j < v; j++) {
        const int h = S >> (j + 1), n = h < NI ? h : NI;
        const uint64_t r = rc[j];
        uint64_t acc[4] = {0, 0, 0, 0};
        for (int i = tid; i < h; i += NI) {
            const uint64_t lo[3] = {ta[i], tb[i], 0}, hi[3] = {ta[i + h], tb[i + h], 0};
            pair_contrib<KIND>(lo, hi, acc);
#pragma unroll
            for (int X = 0; X <= D; X++) acc[X] = m61::fold(acc[X]);
            ta[i] = fold_to(lo[0], hi[0], r);
            tb[i] = fold_to(lo[1], hi[1], r);
        }
        if (tid < n)
#pragma unroll
            for (int X = 0; X <= D; X++) pe[(off + tid) * 3 + X] = acc[X];
        off += n;
        __syncthreads();  // folds of round j visible to round j + 1
    }
    // per-round sums: eight lanes per (round, X), four terms before each fold
    const int ntask = 24 * v;
    for (int task = tid; task < ((ntask + 63) & ~63); task += NI) {  // whole waves iterate together
        uint64_t acc = 0;
        const int q = task >> 3, part = task & 7;
        if (task < ntask) {
            const int j = q / 3, X = q % 3;
            int o = 0;
            for (int jj = 0; jj < j; jj++) o += (S >> (jj + 1)) < NI ? (S >> (jj + 1)) : NI;
            const int n = (S >> (j + 1)) < NI ? (S >> (j + 1)) : NI;
            const uint64_t *src = pe + (size_t)o * 3 + X;
            int e = part;
            for (; e + 24 < n; e += 32) acc = m61::fold(acc + src[3 * e] + src[3 * (e + 8)] + src[3 * (e + 16)] + src[3 * (e + 24)]);
            for (; e < n; e += 8) acc = m61::fold(acc + src[3 * e]);
        }
        acc = m61::fold(acc + __shfl_xor(acc, 1, 64));
        acc = m61::fold(acc + __shfl_xor(acc, 2, 64));
        acc = m61::fold(acc + __shfl_xor(acc, 4, 64));
        if (task < ntask && part == 0) red[q] = m61::canon(acc);
    }
    __syncthreads();
    if (tid < 3 * v) in.tr[in.ev + 3 * in.j0 + tid] = red[tid];
    if (tid == 0 && in.j0 == 0 && v > 0 && in.sum_out >= 0) in.tr[in.sum_out] = m61::add(red[0], red[1]);
    if (tid == 0) {
        if (in.fin0) *in.fin0 = m61::canon(ta[0]);
        if (in.fin1) *in.fin1 = m61::canon(tb[0]);
    }
}

size_t tail_capacity(int) { return kTailMax; }

void launch_tail(int kind, const TailArgs &a, const XJobs &jobs, hipStream_t st)
{
    (void)kind;
    hipLaunchKernelGGL(k_tail<KIND_MATMUL>, dim3(1 + jobs.nslot), dim3(kTailThreads), 0, st, a, jobs);
}

// Kernel attributes set once per process (none needed at present).
void init_kernel_attributes() {}
}  // namespace ra
