// rsetup.hpp -- set-up of the concatenated range check: the constant block
// of the plane rounds and the tables of the rounds over x (xsetup.hpp).  Run
// by extra workgroups of the Gram reduction (planes.hip).
#pragma once
#include "claims.hpp"
#include "common.hpp"
#include "m61.hpp"
#include "xsetup.hpp"

namespace ra {

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

__device__ __forceinline__ uint64_t eq1(uint64_t a, uint64_t b)
{
    return m61::add(m61::mul(a, b), m61::mul(m61::sub(1, a), m61::sub(1, b)));
}

// Workgroup q (of x_setup_blocks) of the set-up of the rounds over x; the
// challenges are first staged in LDS.
__device__ __forceinline__ void x_setup_block(const XSetupArgs &xs, int q)
{
    const int tid = threadIdx.x;
    __shared__ uint64_t rl[64], sl[64], zl[64];
    if (tid < xs.lN) {
        rl[tid] = xs.r[tid];
        sl[tid] = xs.sigx[tid];
        zl[tid] = xs.rho2 ? xs.rho2[tid] : 0;
    }
    __syncthreads();
    x_setup_body(xs, q * blockDim.x + tid, rl, sl, zl);
}

// Claimed sum of the range instance: mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~)
// (l3 with ReLU only); claims = (R~, Rm~, Y~, Z~).  Canonical.
__device__ __forceinline__ uint64_t range_claimed_sum(const uint64_t *lam, uint64_t mu, const uint64_t *cl, int t,
                                                      int relu)
{
    using namespace m61;
    uint64_t H = lmul(lam[0], cl[1]) + lmul(lam[1], fold(cl[0] + (1ull << (t + 1))));
    if (relu) H = fold(H) + lmul(lam[2], cl[2]);
    return canon(lmul(mu, fold(H)));
}

// A deferred witness call's last step (claims.hpp) and, from its claims,
// the claimed sum of the range instance; one workgroup of 256 threads.
constexpr int kClaimsLdsWords = m61::block_sum_words(4, 256) + 12;
__device__ __forceinline__ void witness_claims_block(const RangeConsts &rc, uint64_t *lds)
{
    uint64_t *red = lds, *wres = lds + m61::block_sum_words(4, 256);
    claims_final_block(rc.cj, red, wres);
    if (threadIdx.x == 0) {
        const uint64_t lam[3] = {rc.chal[0], rc.chal[1], rc.chal[2]};
        *rc.range_sum = range_claimed_sum(lam, rc.chal[3], wres + 8, rc.cj.hp.t, rc.cj.hp.relu);
    }
}
__device__ __forceinline__ void witness_claims_block(const RangeConsts &rc)
{
    __shared__ uint64_t lds[kClaimsLdsWords];
    witness_claims_block(rc, lds);
}

// The constant block of the plane rounds (one workgroup of at least 256
// threads); chal points at lambda1: lambda1..3, mu, tau_p (lP), sigma
// (lP + ...).  Every operand is first staged in LDS.
constexpr int kConstsLdsWords = C_WORDS + kMaxPlaneLog + 4 + 2 * kMaxPlaneLog + 3 + 2;
__device__ __forceinline__ void range_consts_block(const RangeConsts &rc, uint64_t *lds)
{
    const uint64_t *chal = rc.chal, *claims = rc.claims;
    const WitParams *prm = rc.prm;
    const int lP = rc.lP, tid = threadIdx.x;
    uint64_t *cst = rc.cst, *range_sum = rc.range_sum;
    using namespace m61;
    uint64_t *c = lds, *eqt = c + C_WORDS, *ch = eqt + kMaxPlaneLog, *cl = ch + 4 + 2 * kMaxPlaneLog;
    int *pv = (int *)(cl + 3);
    const int P = 1 << lP;
    // with the witness's last step deferred (t given), the parameters are the
    // job's and the claimed sum is left to witness_claims_block
    const bool deferred = rc.cj.nblk > 0;
    if (tid < 4 + 2 * lP) ch[tid] = chal[tid];
    if (!deferred && tid >= 64 && tid < 67) cl[tid - 64] = claims[tid - 64];
    if (tid == 128) {
        const WitParams wp = deferred ? rc.cj.hp : *prm;
        pv[0] = wp.s;
        pv[1] = wp.t;
        pv[2] = wp.relu;
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
        for (int i = 0; i < lP - j; i++) {
            const uint64_t z = tau[j + i];
            acc = lmul(acc, ((p >> (lP - j - 1 - i)) & 1) ? z : lsub(1, z));
        }
        c[C_E + idx] = canon(acc);
    }
    if (tid < lP) eqt[tid] = eq1(tau[tid], sig[tid]);  // eq(tau_j, sigma_j)
    __syncthreads();
    // W_{j+1} = W_j bound at sigma_j; w2_j = 2 W_j[p + h] - W_j[p]; the last
    // thread carries K_j = prod_{i<j} eq(tau_i, sigma_i) along
    uint64_t K = 1;
    for (int j = 1; j <= lP; j++) {
        const int h = P >> j;
        const uint64_t *Wj = c + C_W + off_full(P, j);
        for (int p = tid; p < h; p += blockDim.x) {
            c[C_W2 + off_half(P, j) + p] = canon(lsub(2 * Wj[p + h], Wj[p]));
            if (j < lP) c[C_W + off_full(P, j + 1) + p] = canon(Wj[p] + lmul(sig[j - 1], lsub(Wj[p + h], Wj[p])));
        }
        if (tid == 255) {  // (the workgroup has at least 256 threads)
            c[C_K + j - 1] = canon(K);
            c[C_TAU + j - 1] = tau[j - 1];
            K = lmul(K, eqt[j - 1]);
        }
        __syncthreads();
    }
    if (tid == 255) {
        const uint64_t *Wl = c + C_W + off_full(P, lP);
        const uint64_t Wp = fold(Wl[0] + lmul(sig[lP - 1], lsub(Wl[1], Wl[0])));
        c[C_EP] = canon(K);                     // Ep
        c[C_EP + 1] = canon(lsub(lmul(mu, Wp), K));  // c = mu Wp - Ep
        c[C_EP + 2] = canon(Wp);
        c[C_EP + 3] = mu;
        if (!deferred) *range_sum = range_claimed_sum(lam, mu, cl, t, relu);
    }
    __syncthreads();
    for (int i = tid; i < C_WORDS; i += blockDim.x) cst[i] = c[i];
}
__device__ __forceinline__ void range_consts_block(const RangeConsts &rc)
{
    __shared__ uint64_t lds[kConstsLdsWords];
    range_consts_block(rc, lds);
}

}  // namespace ra
