// link.hip -- the gather link between layers.  Sec. III-C chains layers
// through their outputs; a convolution's input is a gather of the previous
// output (im2col: each input entry read by up to kh kw patch positions,
// zero padding; flattening: a permutation).  With A[a] = Z[src[a]] (0 where
// src[a] = -1), the next layer's claim A~(z) at the point z = (r1, rho) of its
// matrix sum-check is
//     A~(z) = sum_y Z[y] W_z[y],   W_z[y] = sum over the a with src[a] = y of eq(z, a),
// a degree-2 sum-check (Sec. II-D) over the entries of Z.  It ends in Z~(y*)
// (a claim on the previous output) and W~_z(y*) (computable from the public
// gather map).
//
// Kernels: the weight table W (one pass over src, modular adds by
// compare-and-swap since several entries read one y), one launch per round
// (evaluate g_j at 0, 1, 2 and fold both tables with that round's
// challenge, which the stream fixes in advance), and a finish launch that
// sums every round's per-block partials into the transcript.
#include <algorithm>

#include "common.hpp"
#include "m61.hpp"

namespace ra {

__global__ __launch_bounds__(256) void k_link_zero(uint64_t *__restrict__ W, uint64_t nz, uint32_t *__restrict__ bad)
{
    if (blockIdx.x == 0 && threadIdx.x == 0) *bad = 0;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nz; i += (uint64_t)gridDim.x * blockDim.x)
        W[i] = 0;
}

// eq(z, a) = E1[a >> lm] E2[a mod 2^lm] (row variables first).  A source
// index outside [-1, nz) is not followed: it sets *bad.
__global__ __launch_bounds__(256) void k_link_weights(const int32_t *__restrict__ src, uint64_t na, int lm,
                                                      const uint64_t *__restrict__ E1, const uint64_t *__restrict__ E2,
                                                      uint64_t nz, unsigned long long *__restrict__ W,
                                                      uint32_t *__restrict__ bad)
{
    const uint64_t cmask = (1ull << lm) - 1;
    for (uint64_t a = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; a < na; a += (uint64_t)gridDim.x * blockDim.x) {
        const int32_t y = src[a];
        if (y < 0) {
            if (y != -1) atomicOr(bad, 1u);
            continue;
        }
        if ((uint64_t)y >= nz) {
            atomicOr(bad, 1u);
            continue;
        }
        const uint64_t v = m61::mul(E1[a >> lm], E2[a & cmask]);
        unsigned long long old = W[y], assumed;
        do {
            assumed = old;
            old = atomicCAS(W + y, assumed, (unsigned long long)m61::add(assumed, v));
        } while (old != assumed);
    }
}

// Round j over tables of 2h entries: g(X) = sum_i T0(X) T1(X) at X = 0, 1, 2
// with T(X) = lo + X (hi - lo), then T[i] <- lo + rho (hi - lo).  The first
// round reads T0 from the int32 table Z.
__global__ __launch_bounds__(256) void k_link_round(const int32_t *__restrict__ Z, uint64_t *__restrict__ T0,
                                                    uint64_t *__restrict__ T1, uint64_t h, int first,
                                                    const uint64_t *__restrict__ rho_p, uint64_t *__restrict__ part)
{
    __shared__ uint64_t red[m61::block_sum_words(3, 256)];
    const uint64_t rho = *rho_p;
    uint64_t g[3] = {0, 0, 0};
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < h; i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t lo0 = first ? m61::from_i32(Z[i]) : T0[i];
        const uint64_t hi0 = first ? m61::from_i32(Z[i + h]) : T0[i + h];
        const uint64_t lo1 = T1[i], hi1 = T1[i + h];
        const uint64_t d0 = m61::sub(hi0, lo0), d1 = m61::sub(hi1, lo1);
        g[0] = m61::add(g[0], m61::mul(lo0, lo1));
        g[1] = m61::add(g[1], m61::mul(hi0, hi1));
        g[2] = m61::add(g[2], m61::mul(m61::add(hi0, d0), m61::add(hi1, d1)));
        T0[i] = m61::add(lo0, m61::mul(rho, d0));
        T1[i] = m61::add(lo1, m61::mul(rho, d1));
    }
    m61::block_sum<3>(g, red);
    if (threadIdx.x == 0)
        for (int q = 0; q < 3; q++) part[3 * (size_t)blockIdx.x + q] = g[q];
}

// One workgroup per global round j < j0 sums that round's partials into
// tr[3 j ..]; workgroup 0 also writes the claim g_1(0) + g_1(1) to fin[0].
__global__ __launch_bounds__(256) void k_link_finish(const uint64_t *__restrict__ part, int vz,
                                                     uint64_t *__restrict__ tr, uint64_t *__restrict__ fin)
{
    __shared__ uint64_t red[m61::block_sum_words(3, 256)];
    const int j = blockIdx.x;
    uint64_t v[3] = {0, 0, 0};
    const int nb = link_blocks(1ull << (vz - 1 - j));
    const uint64_t *p = part + (size_t)j * kLinkMaxBlocks * 3;
    for (int b = threadIdx.x; b < nb; b += blockDim.x)
        for (int q = 0; q < 3; q++) v[q] = m61::add(v[q], p[3 * (size_t)b + q]);
    m61::block_sum<3>(v, red);
    if (threadIdx.x == 0) {
        for (int q = 0; q < 3; q++) tr[3 * (size_t)j + q] = v[q];
        if (j == 0) fin[0] = m61::add(v[0], v[1]);
    }
}

// The last vz - j0 rounds (tables of at most 2^kLinkTailLog entries) in one
// workgroup from LDS: the tables after j0 global rounds (Z itself when j0 =
// 0), every round's sums and fold, then fin[1..3] = Z~(y*), W~(y*) and the
// map's status (and fin[0], the claim, when every round is here).
__global__ __launch_bounds__(256) void k_link_tail(const int32_t *__restrict__ Z, const uint64_t *__restrict__ T0g,
                                                   const uint64_t *__restrict__ Wg, int vz, int j0,
                                                   const uint64_t *__restrict__ rho, uint64_t *__restrict__ tr,
                                                   uint64_t *__restrict__ fin, const uint32_t *__restrict__ bad)
{
    __shared__ uint64_t t0[1 << kLinkTailLog], t1[1 << kLinkTailLog];
    __shared__ uint64_t red[m61::block_sum_words(3, 256)];
    const int v = vz - j0;
    const uint32_t size = 1u << v;
    for (uint32_t i = threadIdx.x; i < size; i += blockDim.x) {
        t0[i] = j0 == 0 ? m61::from_i32(Z[i]) : T0g[i];
        t1[i] = Wg[i];
    }
    __syncthreads();
    uint64_t first = 0;
    for (int j = 0; j < v; j++) {
        const uint32_t h = size >> (j + 1);
        const uint64_t r = rho[j0 + j];
        uint64_t g[3] = {0, 0, 0};
        for (uint32_t i = threadIdx.x; i < h; i += blockDim.x) {  // each thread reads and folds its own i
            const uint64_t lo0 = t0[i], hi0 = t0[i + h], lo1 = t1[i], hi1 = t1[i + h];
            const uint64_t d0 = m61::sub(hi0, lo0), d1 = m61::sub(hi1, lo1);
            g[0] = m61::add(g[0], m61::mul(lo0, lo1));
            g[1] = m61::add(g[1], m61::mul(hi0, hi1));
            g[2] = m61::add(g[2], m61::mul(m61::add(hi0, d0), m61::add(hi1, d1)));
            t0[i] = m61::add(lo0, m61::mul(r, d0));
            t1[i] = m61::add(lo1, m61::mul(r, d1));
        }
        m61::block_sum<3>(g, red);
        if (threadIdx.x == 0) {
            for (int q = 0; q < 3; q++) tr[3 * (size_t)(j0 + j) + q] = g[q];
            if (j == 0) first = m61::add(g[0], g[1]);
        }
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    if (j0 == 0) fin[0] = v > 0 ? first : m61::mul(t0[0], t1[0]);
    fin[1] = t0[0];
    fin[2] = t1[0];
    fin[3] = *bad;
}

// The gathered input itself: A[a] = Z[src[a]], 0 where src[a] = -1.  An
// index outside [-1, nz) is not followed (A[a] = 0); ra_link_prove refuses
// the same map.
__global__ __launch_bounds__(256) void k_link_gather(const int32_t *__restrict__ Z, uint64_t nz,
                                                     const int32_t *__restrict__ src, uint64_t na,
                                                     int32_t *__restrict__ A)
{
    for (uint64_t a = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; a < na; a += (uint64_t)gridDim.x * blockDim.x) {
        const int32_t y = src[a];
        A[a] = (y >= 0 && (uint64_t)y < nz) ? Z[y] : 0;
    }
}

void launch_link_gather(const int32_t *Z, uint64_t nz, const int32_t *src, uint64_t na, int32_t *A, hipStream_t st)
{
    const int nb = (int)std::min<uint64_t>((na + kThreads - 1) / kThreads, 4096);
    hipLaunchKernelGGL(k_link_gather, dim3(nb > 0 ? nb : 1), dim3(kThreads), 0, st, Z, nz, src, na, A);
}

void launch_link(const LinkArgs &a, hipStream_t st)
{
    const uint64_t nz = 1ull << a.vz;
    const int zb = link_blocks(nz);
    hipLaunchKernelGGL(k_link_zero, dim3(zb), dim3(kThreads), 0, st, a.W, nz, a.bad);
    const int wb = (int)std::min<uint64_t>((a.na + kThreads - 1) / kThreads, 2048);
    hipLaunchKernelGGL(k_link_weights, dim3(wb > 0 ? wb : 1), dim3(kThreads), 0, st, a.src, a.na, a.lm, a.E1,
                       a.E2, nz, (unsigned long long *)a.W, a.bad);
    const int j0 = a.vz > kLinkTailLog ? a.vz - kLinkTailLog : 0;  // rounds over the global tables
    for (int j = 0; j < j0; j++) {
        const uint64_t h = 1ull << (a.vz - 1 - j);
        hipLaunchKernelGGL(k_link_round, dim3(link_blocks(h)), dim3(kThreads), 0, st, a.Z, a.T0, a.W, h, j == 0 ? 1 : 0,
                           a.rho + j, a.part + (size_t)j * kLinkMaxBlocks * 3);
    }
    if (j0 > 0)
        hipLaunchKernelGGL(k_link_finish, dim3(j0), dim3(kThreads), 0, st, a.part, a.vz, a.tr, a.fin);
    hipLaunchKernelGGL(k_link_tail, dim3(1), dim3(kThreads), 0, st, a.Z, a.T0, a.W, a.vz, j0, a.rho, a.tr, a.fin,
                       a.bad);
}

}  // namespace ra
