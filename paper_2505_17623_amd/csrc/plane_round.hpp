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

__device__ __forceinline__ void plane_round(const PlaneArgs &pa, int j)
{
    __shared__ uint64_t G[64][65];
    __shared__ uint64_t c[32];           // c_y, y < ny
    __shared__ uint64_t part[96];        // [(combo np + p') ny + y]
    __shared__ uint64_t lin[64];         // [a np + p']
    __shared__ uint64_t contrib[32][6];  // [p'][A0 A1 A2 B0 B1 B2]
    const int tid = threadIdx.x, lP = pa.lP, P = 1 << lP;
    const int ny = 1 << (j - 1), np = P >> j, lo = lP - j, nf = 3 * np * ny;
    const uint64_t *sigma = pa.sigma, *cst = pa.cst;
    for (int i = tid; i < P * P; i += blockDim.x) G[i / P][i % P] = pa.G[(i / P) * 64 + (i % P)];
    for (int y = tid; y < ny; y += blockDim.x) {
        uint64_t a = 1;
        for (int k = 0; k < j - 1; k++) a = m61::mul(a, m61::eq1_bit(sigma[k], (y >> (j - 2 - k)) & 1));
        c[y] = a;
    }
    __syncthreads();
    for (int r = tid; r < nf; r += blockDim.x) {
        const int combo = r / (np * ny), rem = r % (np * ny), p = rem / ny, y = rem % ny;
        const int xa = combo == 1 ? 1 : 0, xb = combo == 0 ? 0 : 1;
        const int qa = (y << (lo + 1)) | (xa << lo) | p;
        uint64_t sacc = 0;
        for (int y2 = 0; y2 < ny; y2++) sacc = m61::add(sacc, m61::mul(c[y2], G[qa][(y2 << (lo + 1)) | (xb << lo) | p]));
        part[r] = m61::mul(c[y], sacc);
    }
    for (int r = tid; r < 2 * np; r += blockDim.x) {
        const int xa = r / np, p = r % np;
        uint64_t sacc = 0;
        for (int y = 0; y < ny; y++) {
            const int q = (y << (lo + 1)) | (xa << lo) | p;
            sacc = m61::add(sacc, m61::mul(c[y], G[q][q]));
        }
        lin[r] = sacc;
    }
    __syncthreads();
    for (int p = tid; p < np; p += blockDim.x) {
        uint64_t Q[3] = {0, 0, 0};
        for (int combo = 0; combo < 3; combo++)
            for (int y = 0; y < ny; y++) Q[combo] = m61::add(Q[combo], part[(combo * np + p) * ny + y]);
        const uint64_t L0 = lin[p], L1 = lin[np + p];
        const uint64_t Q2 = m61::add(m61::sub(m61::mul(4, Q[1]), m61::mul(4, Q[2])), Q[0]);
        const uint64_t L2 = m61::sub(m61::add(L1, L1), L0);
        const int oh = P - (P >> (j - 1));
        const uint64_t e = cst[C_E + oh + p], w2 = cst[C_W2 + oh + p];
        const uint64_t *Wj = cst + C_W + (2 * P - 2 * (P >> (j - 1)));
        uint64_t *o = contrib[p];
        o[0] = m61::mul(e, m61::sub(Q[0], L0));
        o[1] = m61::mul(e, m61::sub(Q[1], L1));
        o[2] = m61::mul(e, m61::sub(Q2, L2));
        o[3] = m61::mul(Wj[p], L0);
        o[4] = m61::mul(Wj[p + np], L1);
        o[5] = m61::mul(w2, L2);
    }
    __syncthreads();
    if (tid == 0) {
        uint64_t A[4] = {0, 0, 0, 0}, B[4] = {0, 0, 0, 0};
        for (int p = 0; p < np; p++)
            for (int X = 0; X < 3; X++) {
                A[X] = m61::add(A[X], contrib[p][X]);
                B[X] = m61::add(B[X], contrib[p][3 + X]);
            }
        // quadratic extension to X = 3: f(3) = f(0) + 3 (f(2) - f(1))
        A[3] = m61::add(A[0], m61::mul(3, m61::sub(A[2], A[1])));
        B[3] = m61::add(B[0], m61::mul(3, m61::sub(B[2], B[1])));
        const uint64_t K = cst[C_K + j - 1], tau = cst[C_TAU + j - 1], mu = cst[C_EP + 3];
        for (int X = 0; X < 4; X++)
            pa.tr[4 * (j - 1) + X] = m61::add(m61::mul(m61::mul(K, m61::eq1_small(tau, X)), A[X]), m61::mul(mu, B[X]));
    }
}

}  // namespace ra
