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
#include "tail.hpp"

namespace ra {

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
        // every load before the accumulated table's clears (a store between
        // the loads would keep the later loads behind it)
        uint64_t v[3][L], vh[L];
#pragma unroll
        for (int q = 0; q < NT; q++)
#pragma unroll
            for (int t = 0; t < L; t++) v[q][t] = (q == 0 && in.acc) ? in.acc[i + t * sub] : T[q][i + t * sub];
        if (in.acc) {
#pragma unroll
            for (int t = 0; t < L; t++) vh[t] = in.acc[(sub << C) + i + t * sub];
#pragma unroll
            for (int t = 0; t < L; t++) {
                in.acc[i + t * sub] = 0;
                in.acc[(sub << C) + i + t * sub] = 0;
                v[0][t] = acc_value(v[0][t], vh[t]);
            }
        }
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
                   const uint64_t *kp, uint64_t *part, int stride, hipStream_t st, uint64_t *acc)
{
    const uint64_t sub = S >> C;
    const int nb = round_blocks(sub);
    const InstArgs a{t0, t1, t2, rho, kp, part, acc};
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

template <int KIND>
__global__ __launch_bounds__(kTailThreads) void k_tail(TailArgs in, XJobs jobs)
{
    __shared__ uint64_t smem[kTailSmem];
    tail_block<KIND>(in, jobs, blockIdx.x, smem);
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
