// xrounds.hip -- the rounds over x of the concatenated range check and of
// the ReLU zero-check (Sec. III-B, Eq. (6)), after the plane variables of
// the range check are bound.  Both instances sum over the same Boolean cube
// with the same equality factor EQ(x) = eq(r, x), r = (r1, r2):
//   range  sum_x EQ(x) (Ep Bx(x)^2 + c Bx(x))          (Bx: bit table bound at sigma_p)
//   ReLU   sum_x EQ(x) (R(x)^2 - Y(x)^2) = sum_x EQ(x) D(x) S(x),   D = R - Y, S = R + Y.
// The range instance binds x to sigma_x, the ReLU instance to rho'.
//
// EQ is never stored.  With x bound to z_<j in round j it equals
//   K_j eq1(r_j, X) eq(r_>j, i),      K_j = prod_{l<j} eq1(r_l, z_l),
// so the round polynomial is K_j eq1(r_j, X) s_j(X) with
//   s_j(X) = sum_i eq(r_>j, i) h(T_X(i))     (T_X = T_lo + X (T_hi - T_lo)),
// a quadratic in X.  The kernels accumulate, per round,
//   range  A_a = sum_i w_i b_a,  Q_a = sum_i w_i b_a^2      (a = 0, 1; Q also at b_2 = 2 b_1 - b_0)
//   ReLU   Z_a = sum_i w_i d_a s_a                          (a = 0, 1, 2)
// with w_i = eq(r_>j, i), five field products per pair and instance; the
// assembly forms s_j(0..2), extrapolates s_j(3) and multiplies by
// K_j eq1(r_j, X).  The weights eq(r_>j, i) come from two small tables of
// suffix eq vectors (a high part and a low part of the variables), so they
// cost one product per thread.  The ReLU tables are kept as D and S; the
// final values give R = (D + S) / 2 and Y = (S - D) / 2.
#include <algorithm>

#include "common.hpp"
#include "m61.hpp"

namespace ra {

// Contributions of one pair with weight w: range to acc[0..5), ReLU to acc[0..3).
__device__ __forceinline__ void range_pair(uint64_t w, uint64_t b0, uint64_t b1, uint64_t *acc)
{
    const uint64_t eb0 = m61::mul(w, b0), eb1 = m61::mul(w, b1);
    const uint64_t eb2 = m61::sub(m61::add(eb1, eb1), eb0), b2 = m61::sub(m61::add(b1, b1), b0);
    acc[0] = m61::add(acc[0], eb0);
    acc[1] = m61::add(acc[1], eb1);
    acc[2] = m61::add(acc[2], m61::mul(eb0, b0));
    acc[3] = m61::add(acc[3], m61::mul(eb1, b1));
    acc[4] = m61::add(acc[4], m61::mul(eb2, b2));
}

__device__ __forceinline__ void relu_pair(uint64_t w, uint64_t d0, uint64_t d1, uint64_t s0, uint64_t s1,
                                          uint64_t *acc)
{
    const uint64_t ed0 = m61::mul(w, d0), ed1 = m61::mul(w, d1);
    const uint64_t ed2 = m61::sub(m61::add(ed1, ed1), ed0), s2 = m61::sub(m61::add(s1, s1), s0);
    acc[0] = m61::add(acc[0], m61::mul(ed0, s0));
    acc[1] = m61::add(acc[1], m61::mul(ed1, s1));
    acc[2] = m61::add(acc[2], m61::mul(ed2, s2));
}

__device__ __forceinline__ uint64_t fold(uint64_t lo, uint64_t hi, uint64_t z)
{
    return m61::add(lo, m61::mul(z, m61::sub(hi, lo)));
}

// Sums of NV values over the 64 lanes of the calling wave, written to
// out[0 .. NV).  Every wave of the block calls it at the same point (it holds
// a block barrier); `lw` is the wave's own NV * 68 words of LDS.
template <int NV>
__device__ __forceinline__ void wave_sums_to(const uint64_t (&v)[NV], uint64_t *lw, uint64_t *out)
{
    constexpr int LS = 68;  // padded stride: 16 lanes read 16 distinct bank pairs
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int q = 0; q < NV; q++) lw[q * LS + lane] = v[q];
    __syncthreads();
    for (int t = lane; t < 4 * NV; t += 64) {  // four lanes per value, 16 entries each
        const uint64_t *src = lw + (t >> 2) * LS + (t & 3);
        uint64_t a0 = 0, a1 = 0;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            a0 = m61::add(a0, src[4 * e]);
            a1 = m61::add(a1, src[4 * e + 4]);
        }
        uint64_t sum = m61::add(a0, a1);
        sum = m61::add(sum, __shfl_xor(sum, 1, 64));
        sum = m61::add(sum, __shfl_xor(sum, 2, 64));
        if ((t & 3) == 0) out[t >> 2] = sum;
    }
}

// ---------------------------------------------------------------------------
// C fused rounds j .. j + C - 1 over tables of S = 2^lS entries (lS = lN - j).
// Sub-cube i (< S' = S / 2^C) is the set of entries i + t S' (t < 2^C), the
// values of the C variables being bound; one thread runs the C rounds on one
// sub-cube in registers and writes the bound value to index i.  The pair
// (u, u + h) of local round c has weight eq(r_{j+c+1 .. j+C-1}, u)
// eq(r_{j+C ..}, i), built from eq(r_{j+C ..}, i) = HS[.] LS[.] by halving.
// With ReLU, waves 0-1 of a block run the range instance and waves 2-3 the
// ReLU instance on the same 128 sub-cubes (so a wave carries half the work);
// without, all four waves run the range instance.  With FIRST the inputs are
// Bx and the integer R, Y; D and S are written.  Each wave writes its sums
// of round c to part + c * stride + 8 unit (range words 0-4, ReLU 5-7).
// ---------------------------------------------------------------------------
template <int C>
__device__ __forceinline__ void x_weights(uint64_t e, const uint64_t *rr, uint64_t (&w)[1 << C])
{
    // round c uses w[(1 << (C-1-c)) - 1 + u] (indices 0 .. 2^C - 2)
    w[0] = e;  // round C - 1 (u empty)
#pragma unroll
    for (int c = C - 2; c >= 0; c--) {
        const int hn = 1 << (C - 1 - c), base = hn - 1, pb = (hn >> 1) - 1;
        // u = (msb, rest): eq1(r_{j+c+1}, msb) times the weight of `rest` one round later
#pragma unroll
        for (int u = 0; u < hn / 2; u++) {
            const uint64_t hi = m61::mul(rr[c + 1], w[pb + u]);
            w[base + hn / 2 + u] = hi;
            w[base + u] = m61::sub(w[pb + u], hi);
        }
    }
}

template <int C, bool FIRST, bool RELU>
__global__ __launch_bounds__(256) void k_xrounds(XArgs a, uint64_t sub, int stride)
{
    constexpr int NL = 1 << C, NPB = RELU ? 128 : 256, NVR = 5 * C, NVZ = 3 * C;
    __shared__ uint64_t lw[4][NVR * 68];
    const int tid = threadIdx.x, wv = tid >> 6;
    const bool zw = RELU && wv >= 2;  // wave-uniform
    const int lt = RELU ? (tid & 127) : tid;
    const int unit = RELU ? blockIdx.x * 2 + (wv & 1) : blockIdx.x * 4 + wv;
    uint64_t accr[C][5], accz[C][3];
#pragma unroll
    for (int c = 0; c < C; c++) {
#pragma unroll
        for (int q = 0; q < 5; q++) accr[c][q] = 0;
#pragma unroll
        for (int q = 0; q < 3; q++) accz[c][q] = 0;
    }
    uint64_t rz[C], rr[C];
#pragma unroll
    for (int c = 0; c < C; c++) {
        rz[c] = zw ? a.rho_z[c] : a.rho_a[c];
        rr[c] = a.r[a.j + c];
    }
    const uint64_t *hs = a.HS + (1ull << (a.lN - a.L - a.j - C));
    const uint64_t *ls = a.LS + (1ull << a.L);
    const uint64_t lmask = (1ull << a.L) - 1;
    for (uint64_t i = (uint64_t)blockIdx.x * NPB + lt; i < sub; i += (uint64_t)gridDim.x * NPB) {
        uint64_t w[NL];
        x_weights<C>(m61::mul(hs[i >> a.L], ls[i & lmask]), rr, w);
        if (!zw) {
            uint64_t b[NL];
#pragma unroll
            for (int t = 0; t < NL; t++) b[t] = a.bx[i + t * sub];
#pragma unroll
            for (int c = 0; c < C; c++) {
                const int h = NL >> (c + 1), base = h - 1;
#pragma unroll
                for (int u = 0; u < h; u++) {
                    range_pair(w[base + u], b[u], b[u + h], accr[c]);
                    b[u] = fold(b[u], b[u + h], rz[c]);
                }
            }
            a.bx[i] = b[0];
        } else {
            uint64_t d[NL], s[NL];
#pragma unroll
            for (int t = 0; t < NL; t++) {
                if (FIRST) {
                    const int64_t R = a.R[i + t * sub], Y = a.Y[i + t * sub];
                    d[t] = m61::from_i64(R - Y);
                    s[t] = m61::from_i64(R + Y);
                } else {
                    d[t] = a.d[i + t * sub];
                    s[t] = a.s[i + t * sub];
                }
            }
#pragma unroll
            for (int c = 0; c < C; c++) {
                const int h = NL >> (c + 1), base = h - 1;
#pragma unroll
                for (int u = 0; u < h; u++) {
                    relu_pair(w[base + u], d[u], d[u + h], s[u], s[u + h], accz[c]);
                    d[u] = fold(d[u], d[u + h], rz[c]);
                    s[u] = fold(s[u], s[u + h], rz[c]);
                }
            }
            a.d[i] = d[0];
            a.s[i] = s[0];
        }
    }
    // per-wave sums; the range waves' layout covers both (ReLU values in the first 3 C)
    uint64_t flat[NVR];
#pragma unroll
    for (int c = 0; c < C; c++)
#pragma unroll
        for (int q = 0; q < 5; q++) flat[c * 5 + q] = zw ? (q < 3 ? accz[c][q] : 0) : accr[c][q];
    __shared__ uint64_t tot[4][NVR];
    wave_sums_to<NVR>(flat, lw[wv], tot[wv]);
    __syncthreads();
    const int lane = tid & 63;
    if (lane < C * 8) {
        const int c = lane >> 3, q = lane & 7;
        uint64_t v;
        if (!zw) v = q < 5 ? tot[wv][c * 5 + q] : 0;
        else v = tot[wv][c * 5 + q - 5];
        if (zw ? q >= 5 : (q < 5 || !RELU)) a.part[(size_t)c * stride + (size_t)unit * 8 + q] = v;
    }
}

int xround_blocks(uint64_t sub, bool relu)
{
    const uint64_t per = relu ? 128 : 256, cap = relu ? kMaxUnits / 2 : kMaxUnits / 4;
    const uint64_t b = (sub + per - 1) / per;
    return (int)(b < cap ? (b ? b : 1) : cap);
}

int xround_units(uint64_t sub, bool relu) { return xround_blocks(sub, relu) * (relu ? 2 : 4); }

void launch_xrounds(int C, bool first, bool relu, const XArgs &a, uint64_t S, int stride, hipStream_t st)
{
    const uint64_t sub = S >> C;
    const dim3 g(xround_blocks(sub, relu)), b(kThreads);
#define RA_X(CC, F, Z) hipLaunchKernelGGL((k_xrounds<CC, F, Z>), g, b, 0, st, a, sub, stride)
#define RA_X_FZ(CC)                      \
    if (first) {                         \
        if (relu) RA_X(CC, true, true);  \
        else RA_X(CC, true, false);      \
    } else {                             \
        if (relu) RA_X(CC, false, true); \
        else RA_X(CC, false, false);     \
    }
    switch (C) {
    case 1: RA_X_FZ(1) break;
    case 2: RA_X_FZ(2) break;
    case 3: RA_X_FZ(3) break;
    default: RA_X_FZ(4) break;
    }
#undef RA_X_FZ
#undef RA_X
}

// ---------------------------------------------------------------------------
// The last v rounds in one workgroup with the tables in LDS.  Round jj pairs
// i and i + h (h = 2^(v-1-jj)) with weight LS[h + i] = eq(r_>j, i).  With
// ReLU the first half of the threads runs the range instance and the second
// half the ReLU instance; thread t of a half (t < min(h, half)) writes its
// sums of round jj to part + jj * stride + 8 t (range words 0-4, ReLU 5-7).
// With FIRST (no global rounds ran) the inputs are Bx and the integer R, Y.
// ---------------------------------------------------------------------------
template <bool RELU>
__global__ __launch_bounds__(kXTailThreads) void k_xtail(XTailArgs a, int first, int stride)
{
    __shared__ uint64_t Tb[kXTailMax], Td[RELU ? kXTailMax : 1], Ts[RELU ? kXTailMax : 1], W[kXTailMax];
    constexpr int NH = RELU ? kXTailThreads / 2 : kXTailThreads;  // threads per instance
    const int tid = threadIdx.x, v = a.v, S = 1 << v;
    const bool zw = RELU && tid >= NH;  // wave-uniform
    const int lt = zw ? tid - NH : tid;
    __shared__ uint64_t zc[2][kXTailLog];  // the rounds' challenges, read once
    if (tid < v) zc[0][tid] = a.rho_a[tid];
    if (RELU && tid >= 64 && tid < 64 + v) zc[1][tid - 64] = a.rho_z[tid - 64];
    for (int i = tid; i < S; i += blockDim.x) {
        Tb[i] = a.bx[i];
        W[i] = a.LS[i];  // heap entries 1 .. S-1 are the tables of sizes S/2 .. 1
        if (RELU) {
            if (first) {
                const int64_t R = a.R[i], Y = a.Y[i];
                Td[i] = m61::from_i64(R - Y);
                Ts[i] = m61::from_i64(R + Y);
            } else {
                Td[i] = a.d[i];
                Ts[i] = a.s[i];
            }
        }
    }
    __syncthreads();
    for (int jj = 0; jj < v; jj++) {
        const int h = S >> (jj + 1);
        const uint64_t z = zc[zw ? 1 : 0][jj];
        if (h > NH / 2) {  // many pairs: one thread per pair
            uint64_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if (!zw) {
                for (int i = lt; i < h; i += NH) {
                    const uint64_t w = W[h + i], b0 = Tb[i], b1 = Tb[i + h];
                    range_pair(w, b0, b1, acc);
                    Tb[i] = fold(b0, b1, z);
                }
            } else {
                for (int i = lt; i < h; i += NH) {
                    const uint64_t w = W[h + i], d0 = Td[i], d1 = Td[i + h], s0 = Ts[i], s1 = Ts[i + h];
                    relu_pair(w, d0, d1, s0, s1, acc + 5);
                    Td[i] = fold(d0, d1, z);
                    Ts[i] = fold(s0, s1, z);
                }
            }
            if (lt < h) {
                uint64_t *o = a.part + (size_t)jj * stride + 8 * (size_t)lt;
                if (!zw) {
#pragma unroll
                    for (int q = 0; q < 5; q++) o[q] = acc[q];
                    if (!RELU)
#pragma unroll
                        for (int q = 5; q < 8; q++) o[q] = 0;
                } else {
#pragma unroll
                    for (int q = 5; q < 8; q++) o[q] = acc[q];
                }
            }
        } else {
            // few pairs: four lanes per pair, each at most two products.
            // Role 0, 1, 2 take the terms at b_0, b_1, b_2 = 2 b_1 - b_0 (range:
            // w b_a and w b_a^2; ReLU: (w d_a) s_a); role 3 folds the tables.
            const int role = lt & 3;
            for (int i = lt >> 2; i < h; i += NH / 4) {
                const uint64_t w = W[h + i];
                uint64_t *o = a.part + (size_t)jj * stride + 8 * (size_t)i;
                if (!zw) {
                    const uint64_t b0 = Tb[i], b1 = Tb[i + h];
                    const uint64_t u = role == 0 ? b0 : role == 1 ? b1 : role == 2 ? m61::sub(m61::add(b1, b1), b0)
                                                                                   : m61::sub(b1, b0);
                    const uint64_t xv = m61::mul(role == 3 ? z : w, u);
                    if (role == 3) {
                        Tb[i] = m61::add(b0, xv);
                    } else {
                        const uint64_t yv = m61::mul(xv, u);
                        if (role < 2) o[role] = xv;  // A_0, A_1
                        o[2 + role] = yv;            // Q_0, Q_1, Q_2
                        if (!RELU && role == 0) o[5] = o[6] = o[7] = 0;
                    }
                } else {
                    const uint64_t d0 = Td[i], d1 = Td[i + h], s0 = Ts[i], s1 = Ts[i + h];
                    const uint64_t u = role == 0 ? d0 : role == 1 ? d1 : role == 2 ? m61::sub(m61::add(d1, d1), d0)
                                                                                   : m61::sub(d1, d0);
                    const uint64_t vv = role == 0 ? s0 : role == 1 ? s1 : role == 2 ? m61::sub(m61::add(s1, s1), s0)
                                                                                    : m61::sub(s1, s0);
                    const uint64_t xv = m61::mul(role == 3 ? z : w, u);
                    const uint64_t yv = m61::mul(role == 3 ? z : xv, vv);
                    if (role == 3) {
                        Td[i] = m61::add(d0, xv);
                        Ts[i] = m61::add(s0, yv);
                    } else {
                        o[5 + role] = yv;  // Z_0, Z_1, Z_2
                    }
                }
            }
        }
        __syncthreads();
    }
    if (tid == 0) {
        *a.fin_b = Tb[0];
        if (RELU) {
            const uint64_t inv2 = 1ull << 60;  // (p + 1) / 2
            *a.fin_r = m61::mul(m61::add(Td[0], Ts[0]), inv2);
            *a.fin_y = m61::mul(m61::sub(Ts[0], Td[0]), inv2);
        }
    }
}

int xtail_units(int h, bool relu)
{
    const int nh = relu ? kXTailThreads / 2 : kXTailThreads;
    return h > nh / 2 ? std::min(h, nh) : h;  // one unit per pair when four lanes share a pair
}

void launch_xtail(bool relu, bool first, const XTailArgs &a, int stride, hipStream_t st)
{
    if (relu)
        hipLaunchKernelGGL(k_xtail<true>, dim3(1), dim3(kXTailThreads), 0, st, a, (int)first, stride);
    else
        hipLaunchKernelGGL(k_xtail<false>, dim3(1), dim3(kXTailThreads), 0, st, a, (int)first, stride);
}

}  // namespace ra
