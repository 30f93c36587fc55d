// tail.hpp -- the last rounds of the matrix product's sum-check instance
// (Sec. II-D, Eq. (4)) in one workgroup, shared by the tail kernel and by the
// extra workgroups of the exact-product launch that run it beside the
// product's tiles.
#pragma once
#include "assemble.hpp"
#include "common.hpp"
#include "m61.hpp"
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

// Entry i of a row binding accumulated by the front launch over a table of
// S entries: lo = acc[i] holds the sum of the chunks' low 32 bits, hi =
// acc[S + i] the sum of their high bits, and the value is lo + 2^32 hi mod p.
// Readers clear both words for the next call, after all their loads.
// Canonical result.
__device__ __forceinline__ uint64_t acc_value(uint64_t lo, uint64_t hi)
{
    return m61::add(m61::canon(lo), m61::rotl(m61::canon(hi), 32));
}

// lo + r (hi - lo), folded.
__device__ __forceinline__ uint64_t fold_to(uint64_t lo, uint64_t hi, uint64_t r)
{
    return m61::fold(lo + m61::lmul(r, m61::lsub(hi, lo)));
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
__device__ __forceinline__ void tail_block(const TailArgs &in, const XJobs &jobs, int blk, uint64_t *smem)
{
    constexpr int D = KindTraits<KIND>::D;
    if (blk > 0) {
        const int q = blk - 1;
        assemble_slot(jobs.s[q], jobs.part + (size_t)q * jobs.stride, jobs.tr, jobs.xc, smem);
        return;
    }
    uint64_t *ta = smem, *tb = ta + kTailMax, *pe = tb + kTailMax, *red = pe + 3 * kTailRounds, *rc = red + 3 * kTailMaxLog;
    const int tid = threadIdx.x, v = in.v, NI = blockDim.x;
    const int S = 1 << v;
    if (tid < v) rc[tid] = in.rho[tid];
    for (int i0 = tid; i0 < S; i0 += 4 * NI) {  // loads first, then the clears of an accumulated table
        uint64_t x[4], xh[4], y[4];
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int i = i0 + q * NI;
            x[q] = i < S ? (in.acc ? in.acc[i] : in.t0[i]) : 0;
            xh[q] = i < S && in.acc ? in.acc[S + i] : 0;
            y[q] = i < S ? in.t1[i] : 0;
        }
        if (in.acc)
#pragma unroll
            for (int q = 0; q < 4; q++)
                if (i0 + q * NI < S) {
                    in.acc[i0 + q * NI] = 0;
                    in.acc[S + i0 + q * NI] = 0;
                    x[q] = acc_value(x[q], xh[q]);
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

}  // namespace ra
