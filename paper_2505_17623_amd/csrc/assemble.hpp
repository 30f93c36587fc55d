// assemble.hpp -- from per-unit partial sums of a round to the round's
// evaluations.  Used by the assembly kernel and by extra workgroups of the
// kernels of the rounds over x (which assemble the rounds of the launch
// before them).
#pragma once
#include "common.hpp"
#include "m61.hpp"

namespace ra {

// eq(r, X) = (1 - X) + r (2X - 1) at X = 0 .. 3, folded.
__device__ __forceinline__ uint64_t eq1_at(uint64_t r, int X)
{
    if (X == 0) return m61::lsub(1, r);
    return m61::lsub(m61::lmul(r, (uint64_t)(2 * X - 1)), (uint64_t)(X - 1));
}

// The constants one evaluation of x round j needs (K_j or K'_j, r_j and the
// range instance's two coefficients), loaded ahead of the sums they scale.
struct XEvalK {
    uint64_t K, r, ep, cc;
};
__device__ __forceinline__ XEvalK x_eval_consts(const XConst &xc, int j, bool zr)
{
    return XEvalK{zr ? xc.Kz[j] : xc.Kr[j], xc.r[j], xc.kp[0], xc.kp[1]};
}

// One evaluation of the round polynomial of x round j (Sec. III-B) from the
// round's eight sums acc = (A0, A1, Q0, Q1, M, Z0, Z1, U), see xrounds.hip.
// The values at X = 2 are A2 = 2 A1 - A0, Q2 = Q0 + 4 (Q1 - M),
// Z2 = 3 Z0 + 6 Z1 - 2 U; the range round is K_j eq1(r_j, X) (Ep Q_X + c A_X),
// the ReLU round (zr) K'_j eq1(r_j, X) Z_X, each extended to X = 3 as a
// quadratic times the linear eq factor.  Canonical result.
__device__ __forceinline__ uint64_t x_round_eval(const uint64_t *acc, const XEvalK &k, int X, bool zr)
{
    using namespace m61;
    const uint64_t lin = lmul(k.K, eq1_at(k.r, X));
    uint64_t f0, f1, f2;
    if (!zr) {
        const uint64_t ep = k.ep, cc = k.cc;
        const uint64_t q2 = lsub(fold(acc[2] + 4 * acc[3]), fold(4 * acc[4]));  // inputs < 2^61
        const uint64_t a2 = lsub(2 * acc[1], acc[0]);
        f0 = fold(lmul(ep, acc[2]) + lmul(cc, acc[0]));
        f1 = fold(lmul(ep, acc[3]) + lmul(cc, acc[1]));
        f2 = fold(lmul(ep, q2) + lmul(cc, a2));
    } else {
        f0 = acc[5];
        f1 = acc[6];
        f2 = lsub(fold(fold(3 * acc[5] + 4 * acc[6]) + 2 * acc[6]), 2 * acc[7]);
    }
    // quadratic: f(3) = f(0) + 3 (f(2) - f(1))
    const uint64_t fx = X == 0 ? f0 : X == 1 ? f1 : X == 2 ? f2 : fold(f0 + lmul(3, lsub(f2, f1)));
    return canon(lmul(lin, fx));
}

// LDS words assemble_slot needs for a block of nt threads.
__host__ __device__ constexpr int assemble_slot_words(int nt) { return m61::block_sum_words(kPartWidth, nt); }

// Reduce one slot's partials p[0 .. nblk width) with the whole block and
// write the round's evaluations.  lds: assemble_slot_words(blockDim.x) words.
__device__ __forceinline__ void assemble_slot(const Slot &sl, const uint64_t *__restrict__ p, uint64_t *tr,
                                              const XConst &xc, uint64_t *lds)
{
    // the evaluating threads' constants, fetched with the partials
    XEvalK ek{};
    if (sl.kind != SLOT_COPY && threadIdx.x < 8) ek = x_eval_consts(xc, sl.round, threadIdx.x >= 4);
    uint64_t acc[kPartWidth] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int nt = blockDim.x, w = sl.width;
    int b = threadIdx.x;
    for (; b + 3 * nt < sl.nblk; b += 4 * nt) {  // four units per thread, loads first, one fold
        uint64_t v[4][kPartWidth];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
            for (int i = 0; i < kPartWidth; i++) v[u][i] = i < w ? p[(size_t)(b + u * nt) * w + i] : 0;
#pragma unroll
        for (int i = 0; i < kPartWidth; i++) acc[i] = m61::fold(acc[i] + v[0][i] + v[1][i] + v[2][i] + v[3][i]);
    }
    for (; b < sl.nblk; b += nt)
        for (int i = 0; i < w; i++) acc[i] = m61::fold(acc[i] + p[(size_t)b * w + i]);
    const uint64_t *tot = m61::block_sum_lds<kPartWidth>(acc, lds);
    const int t = threadIdx.x;
    if (sl.kind == SLOT_COPY) {
        if (t < sl.width) tr[sl.out + t] = tot[t];
        if (t == 0 && sl.sum_out >= 0) tr[sl.sum_out] = m61::add(tot[0], tot[1]);  // claimed sum = g_1(0) + g_1(1)
    } else if (t < 8) {  // four evaluations per instance, one per thread
        const bool zr = t >= 4;
        if (!zr || sl.out2 >= 0) tr[(zr ? sl.out2 : sl.out) + (t & 3)] = x_round_eval(tot, ek, t & 3, zr);
    }
}

}  // namespace ra
