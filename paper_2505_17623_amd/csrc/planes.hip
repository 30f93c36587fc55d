// planes.hip -- the plane rounds of the concatenated range check.
//
// Over the bit table b(q, x) (q = plane, the first log P variables; x the
// output index) the range summand is
//   eq(tau_p, q) EQ(x) b (b - 1) + mu W(q) EQ(x) b,     EQ(x) = eq((r1, r2), x).
// While plane variable j is free and x is still Boolean, the round
// polynomial is g_j(X) = K_j eq(tau_j, X) A_j(X) + mu Bw_j(X) with
//   A_j(X)  = sum_p' e_j[p'] sum_x EQ(x) (b_X^2 - b_X),
//   Bw_j(X) = sum_p' W_j(X, p') sum_x EQ(x) b_X,
// b_X = b(sigma_<j, X, p', x) = sum_y c_y bit_(y, X, p')(x), c_y = eq(sigma_<j, y).
// Every x-sum above is a linear combination of the entries of the Gram
// matrix G[q][q'] = sum_x EQ(x) bit_q(x) bit_q'(x) (its diagonal gives the
// linear terms, since a bit squared is itself).  G is an exact integer
// contraction over x, so it runs on the matrix cores: EQ(x) is split into
// nine 7-bit limbs d_t(x), and G_t = Bits^T diag(d_t) Bits is an int8 x int8
// -> int32 product (v_mfma_i32_32x32x32_i8), recombined as sum_t 2^(7t) G_t
// modulo p.  The same pass writes EQ(x) and the plane-bound table
// Bx(x) = sum_q eq(sigma_p, q) bit_q(x) (eight byte lookups per x), the
// inputs of the rounds over x.
#include "common.hpp"
#include "m61.hpp"

namespace ra {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
constexpr int kLimbs = 9;    // 7-bit limbs of a field element (63 bits)

// Output fragment of v_mfma_i32_32x32x32_i8: lane l, register r holds
// row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
__host__ __device__ constexpr int frag_row(int l, int r) { return 8 * (r / 4) + 4 * (l / 32) + (r % 4); }

// Tile pairs of the symmetric 64 x 64 Gram matrix: (0,0), (0,1), (1,1).
__device__ __forceinline__ int tile_row(int tp, int TP) { return TP == 1 ? 0 : (tp == 2 ? 1 : 0); }
__device__ __forceinline__ int tile_col(int tp, int TP) { return TP == 1 ? 0 : (tp == 0 ? 0 : 1); }

// One x per thread for the per-x outputs; wave `tp` then accumulates tile
// pair tp of the Gram matrix over the block's NX = 64 TP outputs.
template <int TP>
__global__ __launch_bounds__(64 * TP) void k_plane_gram(const uint64_t *__restrict__ bits, uint64_t N, int lk,
                                                        const uint64_t *__restrict__ E1,
                                                        const uint64_t *__restrict__ E2,
                                                        const uint64_t *__restrict__ lut, uint64_t *__restrict__ EQ,
                                                        uint64_t *__restrict__ EQ2, uint64_t *__restrict__ Bx,
                                                        uint64_t *__restrict__ gpart)
{
    constexpr int NX = 64 * TP;
    __shared__ uint64_t s_lut[8 * 256];                 // Bx byte tables
    __shared__ uint64_t s_exp[256];                     // byte -> eight 0x00 / 0xFF bytes
    __shared__ __attribute__((aligned(16))) uint8_t s_d[kLimbs][NX];
    __shared__ uint64_t s_mq[TP][2][64];                // plane-major bit masks per wave
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    for (int i = tid; i < 8 * 256; i += NX) s_lut[i] = lut[i];
    for (int i = tid; i < 256; i += NX) {
        uint64_t e = 0;
        for (int b = 0; b < 8; b++)
            if ((i >> b) & 1) e |= 0xFFull << (8 * b);
        s_exp[i] = e;
    }
    const int pt = tile_row(wv, TP), pt2 = tile_col(wv, TP);
    const int half = lane >> 5;
    const uint64_t kmask = (1ull << lk) - 1;
    const uint64_t nchunks = (N + NX - 1) / NX;
    v16i acc[kLimbs];
#pragma unroll
    for (int t = 0; t < kLimbs; t++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[t][r] = 0;
    __syncthreads();

    // the next chunk's word and eq factors are loaded one iteration ahead, so
    // their latency overlaps the matrix-core work of the current chunk
    uint64_t nw = 0, ne1 = 0, ne2 = 0;
    {
        const uint64_t x = (uint64_t)blockIdx.x * NX + tid;
        if (x < N) {
            nw = bits[x];
            ne1 = E1[x >> lk];
            ne2 = E2[x & kmask];
        }
    }
    for (uint64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
        const uint64_t x = ch * NX + tid;
        const bool valid = x < N;
        const uint64_t w = nw, e1 = ne1, e2 = ne2;
        {
            const uint64_t xn = (ch + gridDim.x) * NX + tid;
            if (xn < N) {
                nw = bits[xn];
                ne1 = E1[xn >> lk];
                ne2 = E2[xn & kmask];
            }
        }
        uint64_t eqx = 0;
        if (valid) {
            eqx = m61::mul(e1, e2);
            EQ[x] = eqx;
            if (EQ2) EQ2[x] = eqx;
        }
        uint64_t bx = 0;
#pragma unroll
        for (int b = 0; b < 8; b++) bx = m61::add(bx, s_lut[b * 256 + ((w >> (8 * b)) & 255)]);
        if (valid) Bx[x] = bx;
#pragma unroll
        for (int t = 0; t < kLimbs; t++) s_d[t][tid] = (uint8_t)((eqx >> (7 * t)) & 127);
        // transpose this wave's 64 words: lane l keeps the masks of planes l%32 and l%32 + 32
        uint64_t m0 = 0, m1 = 0;
#pragma unroll
        for (int q = 0; q < (TP == 1 ? 32 : 64); q++) {
            const uint64_t m = __ballot((int)((w >> q) & 1));
            if ((lane & 31) == (q & 31)) {
                if (q < 32) m0 = m;
                else m1 = m;
            }
        }
        s_mq[wv][0][lane] = m0;
        if (TP > 1) s_mq[wv][1][lane] = m1;
        __syncthreads();
#pragma unroll
        for (int g = 0; g < TP; g++) {
            const uint64_t ma = s_mq[g][pt][lane], mb = s_mq[g][pt2][lane];
#pragma unroll
            for (int ks = 0; ks < 2; ks++) {
                // 32 x's per step: half 0 of the lanes carries x 0..15, half 1 x 16..31,
                // in the same byte order for both operands
                const int sh = 32 * ks + 16 * half;
                const uint32_t sa = (uint32_t)(ma >> sh) & 0xFFFF, sb = (uint32_t)(mb >> sh) & 0xFFFF;
                const uint64_t ea0 = s_exp[sa & 255], ea1 = s_exp[sa >> 8];
                const uint64_t eb0 = s_exp[sb & 255], eb1 = s_exp[sb >> 8];
                const v4i A = {(int)((uint32_t)ea0 & 0x01010101u), (int)((uint32_t)(ea0 >> 32) & 0x01010101u),
                               (int)((uint32_t)ea1 & 0x01010101u), (int)((uint32_t)(ea1 >> 32) & 0x01010101u)};
                const v4i Bm = {(int)(uint32_t)eb0, (int)(uint32_t)(eb0 >> 32), (int)(uint32_t)eb1,
                                (int)(uint32_t)(eb1 >> 32)};
                const int xo = 64 * g + sh;
#pragma unroll
                for (int t = 0; t < kLimbs; t++) {
                    const v4i D = *(const v4i *)&s_d[t][xo];
                    acc[t] = __builtin_amdgcn_mfma_i32_32x32x32_i8(A, Bm & D, acc[t], 0, 0, 0);
                }
            }
        }
        __syncthreads();
    }
    // recombine the limbs modulo p and write this block's partial tile
    uint64_t *out = gpart + ((size_t)blockIdx.x * TP + wv) * 1024;
#pragma unroll
    for (int r = 0; r < 16; r++) {
        uint64_t f = 0;
#pragma unroll
        for (int t = 0; t < kLimbs; t++) f = m61::add(f, m61::mul((uint64_t)(uint32_t)acc[t][r], 1ull << (7 * t)));
        out[lane * 16 + r] = f;
    }
}

// Sum of the blocks' partial tiles, written as G[q][q'] (64 x 64, both
// triangles).  Each block covers 64 tile entries; its four waves split the
// partial blocks and combine through LDS.
__global__ __launch_bounds__(256) void k_gram_reduce(const uint64_t *__restrict__ gpart, int nblk, int TP,
                                                     uint64_t *__restrict__ G)
{
    __shared__ uint64_t red[4][64];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, entries = TP * 1024;
    const int e = blockIdx.x * 64 + lane;
    uint64_t a[4] = {0, 0, 0, 0};
    int b = wid;
    for (; b + 12 < nblk; b += 16)
#pragma unroll
        for (int u = 0; u < 4; u++) a[u] = m61::add(a[u], gpart[(size_t)(b + 4 * u) * entries + e]);
    for (; b < nblk; b += 4) a[0] = m61::add(a[0], gpart[(size_t)b * entries + e]);
    red[wid][lane] = m61::add(m61::add(a[0], a[1]), m61::add(a[2], a[3]));
    __syncthreads();
    if (wid != 0) return;
    const uint64_t v = m61::add(m61::add(red[0][lane], red[1][lane]), m61::add(red[2][lane], red[3][lane]));
    const int tp = e >> 10, l = (e & 1023) >> 4, r = e & 15;
    const int q = 32 * tile_row(tp, TP) + frag_row(l, r), q2 = 32 * tile_col(tp, TP) + (l & 31);
    G[q * 64 + q2] = v;
    G[q2 * 64 + q] = v;  // symmetric (the same value when the tile is diagonal)
}

// Round polynomials of the plane rounds from G.  One block of 256 threads;
// the rounds are independent given G, so all of them are evaluated at once.
// For round j (ny = 2^(j-1) bound-variable patterns y, np = P / 2^j suffixes p'):
//   Q_ab(p') = sum_{y,y'} c_y c_y' G[(y,a,p')][(y',b,p')],  L_a(p') = sum_y c_y G[(y,a,p')][(y,a,p')],
// giving sum_x EQ b_a b_b and sum_x EQ b_a; b_2 = 2 b_1 - b_0 is extrapolated.
__global__ __launch_bounds__(256) void k_plane_assemble(const uint64_t *__restrict__ Gg, int lP,
                                                        const uint64_t *__restrict__ sigma,
                                                        const uint64_t *__restrict__ cst, uint64_t *__restrict__ tr)
{
    __shared__ uint64_t G[64][65];
    __shared__ uint64_t c[64];              // round j's c_y at (1 << (j - 1)) - 1 + y
    __shared__ uint64_t part[6][96];        // [j][(combo np + p') ny + y]
    __shared__ uint64_t lin[6][64];         // [j][a np + p']
    __shared__ uint64_t contrib[6][32][6];  // [j][p'][A0 A1 A2 B0 B1 B2]
    const int tid = threadIdx.x, P = 1 << lP, nf = 3 * (P / 2);
    for (int i = tid; i < P * P; i += blockDim.x) G[i / P][i % P] = Gg[(i / P) * 64 + (i % P)];
    for (int i = tid; i < P - 1; i += blockDim.x) {
        int j = 1;
        while (i >= (1 << j) - 1) j++;
        const int y = i - ((1 << (j - 1)) - 1);
        uint64_t a = 1;
        for (int k = 0; k < j - 1; k++) a = m61::mul(a, m61::eq1_bit(sigma[k], (y >> (j - 2 - k)) & 1));
        c[i] = a;
    }
    __syncthreads();
    for (int t = tid; t < lP * nf; t += blockDim.x) {
        const int j = t / nf + 1, r = t % nf, ny = 1 << (j - 1), np = P >> j, lo = lP - j;
        const int combo = r / (np * ny), rem = r % (np * ny), p = rem / ny, y = rem % ny;
        const int xa = combo == 1 ? 1 : 0, xb = combo == 0 ? 0 : 1;
        const uint64_t *cj = c + (ny - 1);
        const int qa = (y << (lo + 1)) | (xa << lo) | p;
        uint64_t sacc = 0;
        for (int y2 = 0; y2 < ny; y2++) sacc = m61::add(sacc, m61::mul(cj[y2], G[qa][(y2 << (lo + 1)) | (xb << lo) | p]));
        part[j - 1][r] = m61::mul(cj[y], sacc);
    }
    for (int t = tid; t < lP * P; t += blockDim.x) {
        const int j = t / P + 1, r = t % P, ny = 1 << (j - 1), np = P >> j, lo = lP - j;
        if (r >= 2 * np) continue;
        const int xa = r / np, p = r % np;
        const uint64_t *cj = c + (ny - 1);
        uint64_t sacc = 0;
        for (int y = 0; y < ny; y++) {
            const int q = (y << (lo + 1)) | (xa << lo) | p;
            sacc = m61::add(sacc, m61::mul(cj[y], G[q][q]));
        }
        lin[j - 1][r] = sacc;
    }
    __syncthreads();
    for (int t = tid; t < lP * 32; t += blockDim.x) {
        const int j = t / 32 + 1, p = t % 32, ny = 1 << (j - 1), np = P >> j;
        if (p >= np) continue;
        uint64_t Q[3] = {0, 0, 0};
        for (int combo = 0; combo < 3; combo++)
            for (int y = 0; y < ny; y++) Q[combo] = m61::add(Q[combo], part[j - 1][(combo * np + p) * ny + y]);
        const uint64_t L0 = lin[j - 1][p], L1 = lin[j - 1][np + p];
        const uint64_t Q2 = m61::add(m61::sub(m61::mul(4, Q[1]), m61::mul(4, Q[2])), Q[0]);
        const uint64_t L2 = m61::sub(m61::add(L1, L1), L0);
        const int oh = P - (P >> (j - 1));
        const uint64_t e = cst[C_E + oh + p], w2 = cst[C_W2 + oh + p];
        const uint64_t *Wj = cst + C_W + (2 * P - 2 * (P >> (j - 1)));
        uint64_t *o = contrib[j - 1][p];
        o[0] = m61::mul(e, m61::sub(Q[0], L0));
        o[1] = m61::mul(e, m61::sub(Q[1], L1));
        o[2] = m61::mul(e, m61::sub(Q2, L2));
        o[3] = m61::mul(Wj[p], L0);
        o[4] = m61::mul(Wj[p + np], L1);
        o[5] = m61::mul(w2, L2);
    }
    __syncthreads();
    if (tid < lP) {
        const int j = tid + 1, np = P >> j;
        uint64_t A[4] = {0, 0, 0, 0}, B[4] = {0, 0, 0, 0};
        for (int p = 0; p < np; p++)
            for (int X = 0; X < 3; X++) {
                A[X] = m61::add(A[X], contrib[j - 1][p][X]);
                B[X] = m61::add(B[X], contrib[j - 1][p][3 + X]);
            }
        // quadratic extension to X = 3: f(3) = f(0) + 3 (f(2) - f(1))
        A[3] = m61::add(A[0], m61::mul(3, m61::sub(A[2], A[1])));
        B[3] = m61::add(B[0], m61::mul(3, m61::sub(B[2], B[1])));
        const uint64_t K = cst[C_K + j - 1], tau = cst[C_TAU + j - 1], mu = cst[C_EP + 3];
        for (int X = 0; X < 4; X++)
            tr[4 * (j - 1) + X] = m61::add(m61::mul(m61::mul(K, m61::eq1_small(tau, X)), A[X]), m61::mul(mu, B[X]));
    }
}

int plane_gram_tiles(int lP) { return lP > 5 ? 3 : 1; }

int plane_gram_blocks(uint64_t N, int lP)
{
    const int TP = plane_gram_tiles(lP);
    const uint64_t chunks = (N + 64 * TP - 1) / (64 * TP);
    return (int)(chunks < 256 ? chunks : 256);
}

void launch_plane_gram(int lP, const uint64_t *bits, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2,
                       const uint64_t *lut, uint64_t *EQ, uint64_t *EQ2, uint64_t *Bx, uint64_t *gpart,
                       uint64_t *gsum, hipStream_t st)
{
    const int TP = plane_gram_tiles(lP), nb = plane_gram_blocks(N, lP);
    if (TP == 1)
        hipLaunchKernelGGL(k_plane_gram<1>, dim3(nb), dim3(64), 0, st, bits, N, lk, E1, E2, lut, EQ, EQ2, Bx, gpart);
    else
        hipLaunchKernelGGL(k_plane_gram<3>, dim3(nb), dim3(192), 0, st, bits, N, lk, E1, E2, lut, EQ, EQ2, Bx, gpart);
    hipLaunchKernelGGL(k_gram_reduce, dim3(TP * 16), dim3(256), 0, st, (const uint64_t *)gpart, nb, TP, gsum);
}

void launch_plane_assemble(int lP, const uint64_t *gsum, const uint64_t *sigma, const uint64_t *cst, uint64_t *tr,
                           hipStream_t st)
{
    hipLaunchKernelGGL(k_plane_assemble, dim3(1), dim3(256), 0, st, gsum, lP, sigma, cst, tr);
}

}  // namespace ra
