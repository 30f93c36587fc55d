// plane_round.hpp -- round polynomials of the plane rounds of the
// concatenated range check from the Gram matrix G (planes.hip): one
// workgroup of 256 threads per round.
//
// For round j (ny = 2^(j-1) bound-variable patterns y, np = P / 2^j
// suffixes p'):
//   Q_ab(p') = sum_{y,y'} c_y c_y' G[(y,a,p')][(y',b,p')],  L_a(p') = sum_y c_y G[(y,a,p')][(y,a,p')],
// with c_y = eq(sigma_<j, y), give sum_x EQ b_a b_b and sum_x EQ b_a; b_2 =
// 2 b_1 - b_0 is extrapolated.  With e_j, W_j, K_j, tau_j from the constant
// block (sumcheck.hip) the round polynomial is
//   g_j(X) = K_j eq(tau_j, X) A_j(X) + mu Bw_j(X),
// A_j and Bw_j quadratic in X (evaluated at 0, 1, 2, extended to 3).
#pragma once
#include "common.hpp"
#include "m61.hpp"

namespace ra {

// LDS words plane_round uses.
constexpr int kPlaneRoundWords = 64 * 65 + 32 + 96 + 64 + 96 + 32 * 6 + 8 + kMaxPlaneLog;

// LDS words of a workgroup of 256 threads that assembles a slot
// (assemble.hpp) or evaluates a plane round.
constexpr int kJobLdsWords = kPlaneRoundWords > m61::block_sum_words(kPartWidth, 256)
                                 ? kPlaneRoundWords
                                 : m61::block_sum_words(kPartWidth, 256);

// lds: kPlaneRoundWords words; 256 threads.  Sums of products are formed from
// loose residues (m61.hpp) and spread over the threads so that no thread
// runs a long dependent chain.
__device__ __forceinline__ void plane_round(const PlaneArgs &pa, int j, uint64_t *lds)
{
    using namespace m61;
    uint64_t(*G)[65] = (uint64_t(*)[65])lds;
    uint64_t *c = lds + 64 * 65;             // c_y, y < ny
    uint64_t *part = c + 32;                 // [(combo np + p') ny + y]
    uint64_t *lin = part + 96;               // [a np + p']
    uint64_t *Qs = lin + 64;                 // [combo np + p']
    uint64_t(*contrib)[6] = (uint64_t(*)[6])(Qs + 96);  // [p'][A0 A1 A2 B0 B1 B2]
    uint64_t *col = Qs + 96 + 32 * 6;        // column sums of contrib
    uint64_t *sg = col + 8;                  // sigma_<j
    const int tid = threadIdx.x, lP = pa.lP, P = 1 << lP;
    const int ny = 1 << (j - 1), np = P >> j, lo = lP - j, nf = 3 * np * ny;
    const uint64_t *cst = pa.cst;
    // operands of the last steps, fetched before the first wait
    const int oh = P - (P >> (j - 1));
    const uint64_t *Wj = cst + C_W + (2 * P - 2 * (P >> (j - 1)));
    uint64_t e = 0, w2 = 0, wa = 0, wb = 0, K = 0, tau = 0, mu = 0;
    if (tid < np) {
        e = cst[C_E + oh + tid];
        w2 = cst[C_W2 + oh + tid];
        wa = Wj[tid];
        wb = Wj[tid + np];
    }
    if (tid < 4) {
        K = cst[C_K + j - 1];
        tau = cst[C_TAU + j - 1];
        mu = cst[C_EP + 3];
    }
    if (tid < j - 1) sg[tid] = pa.sigma[tid];
    // the whole 64 x 64 word matrix (entries past P are not used), every load
    // of a thread issued before the first store
    for (int i0 = tid; i0 < 64 * 64; i0 += 16 * blockDim.x) {
        uint64_t v[16];
#pragma unroll
        for (int q = 0; q < 16; q++) {
            const int i = i0 + q * blockDim.x;
            v[q] = i < 64 * 64 ? pa.G[i] : 0;
        }
#pragma unroll
        for (int q = 0; q < 16; q++) {
            const int i = i0 + q * blockDim.x;
            if (i < 64 * 64) G[i >> 6][i & 63] = v[q];
        }
    }
    __syncthreads();
    for (int y = tid; y < ny; y += blockDim.x) {  // c_y = eq(sigma_<j, y)
        uint64_t a = 1;
        for (int k = 0; k < j - 1; k++) {
            const uint64_t z = sg[k];
            a = lmul(a, ((y >> (j - 2 - k)) & 1) ? z : lsub(1, z));
        }
        c[y] = a;
    }
    __syncthreads();
    if (tid < 2 * nf) {
        // part[r] = c_y sum_y2 c_y2 G[(y, xa, p')][(y2, xb, p')], two lanes per r
        const int r = tid >> 1, half = tid & 1;
        const int combo = r / (np * ny), rem = r % (np * ny), p = rem / ny, y = rem % ny;
        const int xa = combo == 1 ? 1 : 0, xb = combo == 0 ? 0 : 1;
        const int qa = (y << (lo + 1)) | (xa << lo) | p;
        const int hn = (ny + 1) >> 1, y0 = half * hn, y1 = ny < y0 + hn ? ny : y0 + hn;
        uint64_t acc = 0;
        int y2 = y0;
        for (; y2 + 3 < y1; y2 += 4) {
            const uint64_t t0 = lmul(c[y2], G[qa][(y2 << (lo + 1)) | (xb << lo) | p]);
            const uint64_t t1 = lmul(c[y2 + 1], G[qa][((y2 + 1) << (lo + 1)) | (xb << lo) | p]);
            const uint64_t t2 = lmul(c[y2 + 2], G[qa][((y2 + 2) << (lo + 1)) | (xb << lo) | p]);
            const uint64_t t3 = lmul(c[y2 + 3], G[qa][((y2 + 3) << (lo + 1)) | (xb << lo) | p]);
            acc = fold(acc + fold(t0 + t1 + t2 + t3));
        }
        for (; y2 < y1; y2++) acc = fold(acc + lmul(c[y2], G[qa][(y2 << (lo + 1)) | (xb << lo) | p]));
        acc = fold(acc + __shfl_xor(acc, 1, 64));
        if (half == 0) part[r] = lmul(c[y], acc);
    } else if (tid >= 192 && tid - 192 < 2 * np) {
        // lin[r] = sum_y c_y G[q][q], q = (y, xa, p')
        const int r = tid - 192, xa = r / np, p = r % np;
        uint64_t acc = 0;
        for (int y = 0; y < ny; y++) {
            const int q = (y << (lo + 1)) | (xa << lo) | p;
            acc = fold(acc + lmul(c[y], G[q][q]));
        }
        lin[r] = acc;
    }
    __syncthreads();
    if (tid < 3 * np) {  // Q[combo][p'] = sum_y part
        const uint64_t *src = part + tid * ny;
        uint64_t acc = 0;
        int y = 0;
        for (; y + 3 < ny; y += 4) acc = fold(acc + src[y] + src[y + 1] + src[y + 2] + src[y + 3]);
        for (; y < ny; y++) acc = fold(acc + src[y]);
        Qs[tid] = acc;
    }
    __syncthreads();
    if (tid < np) {
        const int p = tid;
        const uint64_t Q0 = Qs[p], Q1 = Qs[np + p], Qx = Qs[2 * np + p];
        const uint64_t L0 = lin[p], L1 = lin[np + p];
        const uint64_t Q2 = lsub(fold(Q0 + 4 * Q1), fold(4 * Qx));  // (2 b1 - b0)^2 = 4 b1 b1 - 4 b0 b1 + b0 b0
        const uint64_t L2 = lsub(2 * L1, L0);
        uint64_t *o = contrib[p];
        o[0] = lmul(e, lsub(Q0, L0));
        o[1] = lmul(e, lsub(Q1, L1));
        o[2] = lmul(e, lsub(Q2, L2));
        o[3] = lmul(wa, L0);
        o[4] = lmul(wb, L1);
        o[5] = lmul(w2, L2);
    }
    __syncthreads();
    if (tid < 6) {  // column sums over p'
        uint64_t acc = 0;
        for (int p = 0; p < np; p++) acc = fold(acc + contrib[p][tid]);
        col[tid] = acc;
    }
    __syncthreads();
    if (tid < 4) {  // g_j(X) = K_j eq(tau_j, X) A(X) + mu B(X), quadratics extended to X = 3
        const int X = tid;
        const uint64_t *A = col, *B = col + 3;
        const uint64_t ax = X < 3 ? A[X] : fold(A[0] + lmul(3, lsub(A[2], A[1])));
        const uint64_t bx = X < 3 ? B[X] : fold(B[0] + lmul(3, lsub(B[2], B[1])));
        const uint64_t eqx = X == 0 ? lsub(1, tau) : lsub(lmul(tau, (uint64_t)(2 * X - 1)), (uint64_t)(X - 1));
        pa.tr[4 * (j - 1) + X] = canon(lmul(lmul(K, eqx), ax) + lmul(mu, bx));
    }
}

}  // namespace ra
