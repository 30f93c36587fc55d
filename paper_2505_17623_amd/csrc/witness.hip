// witness.hip -- eq tables, exact integer matrix product, multilinear binding
// of matrix sides, and the rescale / ReLU / bit-plane witness.
#include "claims.hpp"
#include "common.hpp"
#include "m61.hpp"
#include "ra.h"

namespace ra {

typedef int v4i __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// eq table (Eq. (1) / chi vector of Sec. II-C):
//   out[i] = prod_j (z_j i_j + (1 - z_j)(1 - i_j)),  i_1 = MSB of i.
// ---------------------------------------------------------------------------
// Entries blk*256 + tid, stepping by nblk*256, of the table of the point zl
// (in LDS, v variables).
__device__ __forceinline__ void eq_table_entries(const uint64_t *zl, int v, uint64_t *__restrict__ out, int blk,
                                                 int nblk)
{
    const uint64_t n = 1ull << v;
    for (uint64_t i = (uint64_t)blk * blockDim.x + threadIdx.x; i < n; i += (uint64_t)nblk * blockDim.x) {
        uint64_t acc = 1;
        for (int j = 0; j < v; j++) {
            const uint64_t zj = zl[j];
            acc = m61::lmul(acc, ((i >> (v - 1 - j)) & 1) ? zj : m61::lsub(1, zj));
        }
        out[i] = m61::canon(acc);
    }
}

// Workgroups below nb1 fill the first table (point z1, v1 variables), the
// others the second; the point is staged in LDS first.
__global__ __launch_bounds__(256) void k_eq_tables(const uint64_t *__restrict__ z1, int v1, uint64_t *__restrict__ out1,
                                                   int nb1, const uint64_t *__restrict__ z2, int v2,
                                                   uint64_t *__restrict__ out2)
{
    __shared__ uint64_t zl[64];
    const bool second = (int)blockIdx.x >= nb1;
    const uint64_t *z = second ? z2 : z1;
    const int v = second ? v2 : v1, blk = second ? blockIdx.x - nb1 : blockIdx.x;
    const int nblk = second ? gridDim.x - nb1 : nb1;
    uint64_t *out = second ? out2 : out1;
    if ((int)threadIdx.x < v) zl[threadIdx.x] = z[threadIdx.x];
    __syncthreads();
    eq_table_entries(zl, v, out, blk, nblk);
}

// The same table from a point passed by value (no device copy of the point).
__global__ __launch_bounds__(256) void k_eq_table_val(EqPoint pt, uint64_t *__restrict__ out)
{
    __shared__ uint64_t zl[64];
    if ((int)threadIdx.x < pt.v) zl[threadIdx.x] = pt.z[threadIdx.x];
    __syncthreads();
    eq_table_entries(zl, pt.v, out, blockIdx.x, gridDim.x);
}

static int eq_blocks(int v)
{
    const uint64_t n = 1ull << v;
    return (int)((n + kThreads - 1) / kThreads < 4096 ? (n + kThreads - 1) / kThreads : 4096);
}

void launch_eq_table(const uint64_t *z, int v, uint64_t *out, hipStream_t st)
{
    hipLaunchKernelGGL(k_eq_tables, dim3(eq_blocks(v)), dim3(kThreads), 0, st, z, v, out, eq_blocks(v), z, v, out);
}

void launch_eq_table_val(const EqPoint &pt, uint64_t *out, hipStream_t st)
{
    hipLaunchKernelGGL(k_eq_table_val, dim3(eq_blocks(pt.v)), dim3(kThreads), 0, st, pt, out);
}

void launch_eq_tables(const uint64_t *z1, int v1, uint64_t *out1, const uint64_t *z2, int v2, uint64_t *out2,
                      hipStream_t st)
{
    const int nb1 = eq_blocks(v1), nb2 = eq_blocks(v2);
    hipLaunchKernelGGL(k_eq_tables, dim3(nb1 + nb2), dim3(kThreads), 0, st, z1, v1, out1, nb1, z2, v2, out2);
}

// ---------------------------------------------------------------------------
// Binding one side of a matrix with an eq table (Eq. (4): a~(r1, l) is the
// r1-row combination of A, b~(l, r2) the r2-column combination of B).
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ uint64_t term(uint64_t e, T a);
template <> __device__ __forceinline__ uint64_t term<int16_t>(uint64_t e, int16_t a) { return m61::mul_small(e, a); }
template <> __device__ __forceinline__ uint64_t term<int32_t>(uint64_t e, int32_t a) { return m61::mul_small(e, a); }
template <> __device__ __forceinline__ uint64_t term<int64_t>(uint64_t e, int64_t a)
{
    return m61::mul(e, m61::from_i64(a));
}
template <> __device__ __forceinline__ uint64_t term<uint64_t>(uint64_t e, uint64_t a) { return m61::mul(e, a); }

// Rows are split into chunks; a block reduces one chunk for 64 columns (four
// waves over interleaved rows, then through LDS), a second pass sums chunks.
int bind_rows_chunks(uint32_t rows, uint32_t cols)
{
    const uint32_t groups = (cols + 63) / 64;
    uint32_t nch = 1024 / groups;
    if (nch > 128) nch = 128;
    if (nch > rows / 4) nch = rows / 4;
    return nch ? (int)nch : 1;
}

template <typename T>
__global__ __launch_bounds__(256) void k_bind_rows(const T *__restrict__ A, uint32_t rows, uint32_t cols,
                                                   const uint64_t *__restrict__ E, uint32_t per_chunk,
                                                   uint64_t *__restrict__ part)
{
    __shared__ uint64_t red[4][64];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const uint32_t c = blockIdx.x * 64 + lane;
    const uint32_t r0 = blockIdx.y * per_chunk;
    const uint32_t r1 = r0 + per_chunk < rows ? r0 + per_chunk : rows;
    uint64_t acc = 0;
    if (c < cols)
        for (uint32_t r = r0 + wid; r < r1; r += 4) acc = m61::add(acc, term<T>(E[r], A[(size_t)r * cols + c]));
    red[wid][lane] = acc;
    __syncthreads();
    if (wid == 0 && c < cols)
        part[(size_t)blockIdx.y * cols + c] =
            m61::add(m61::add(red[0][lane], red[1][lane]), m61::add(red[2][lane], red[3][lane]));
}

// The chunk sums of a row binding: 64 columns per workgroup, four threads
// per column (consecutive lanes), four terms added before each fold.
__device__ __forceinline__ void sum_chunks_block(const ChunkSum &cs, uint32_t blk)
{
    const uint32_t c = blk * 64 + (threadIdx.x >> 2), cols = cs.cols;
    const int q0 = threadIdx.x & 3, nch = cs.nch;
    const uint64_t *p = cs.part;
    uint64_t acc = 0;
    if (c < cols) {
        int q = q0;
        for (; q + 12 < nch; q += 16)
            acc = m61::fold(acc + p[(size_t)q * cols + c] + p[(size_t)(q + 4) * cols + c] +
                            p[(size_t)(q + 8) * cols + c] + p[(size_t)(q + 12) * cols + c]);
        for (; q < nch; q += 4) acc = m61::fold(acc + p[(size_t)q * cols + c]);
    }
    acc = m61::fold(acc + __shfl_xor(acc, 1, 64));
    acc = m61::fold(acc + __shfl_xor(acc, 2, 64));
    if (c < cols && q0 == 0) cs.out[c] = m61::canon(acc);
}

__global__ __launch_bounds__(256) void k_sum_chunks(ChunkSum cs) { sum_chunks_block(cs, blockIdx.x); }

static int sum_chunks_blocks(uint32_t cols) { return (int)((cols + 63) / 64); }

template <typename T>
__global__ __launch_bounds__(256) void k_bind_cols(const T *__restrict__ B, uint32_t rows, uint32_t cols,
                                                   const uint64_t *__restrict__ E, uint64_t *__restrict__ out)
{
    const uint32_t row = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;  // one wave per row
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;                                          // wave-uniform
    uint64_t acc = 0;
    for (uint32_t c = lane; c < cols; c += 64) acc = m61::add(acc, term<T>(E[c], B[(size_t)row * cols + c]));
    acc = m61::wave_sum(acc);
    if (lane == 0) out[row] = acc;
}

void launch_bind_rows(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E, uint64_t *scratch,
                      uint64_t *out, hipStream_t st)
{
    const int nch = bind_rows_chunks(rows, cols);
    const uint32_t per = (rows + nch - 1) / nch;
    dim3 grid((cols + 63) / 64, nch);
    switch (dtype) {
    case RA_I16: hipLaunchKernelGGL(k_bind_rows<int16_t>, grid, dim3(256), 0, st, (const int16_t *)T, rows, cols, E, per, scratch); break;
    case RA_I32: hipLaunchKernelGGL(k_bind_rows<int32_t>, grid, dim3(256), 0, st, (const int32_t *)T, rows, cols, E, per, scratch); break;
    case RA_I64: hipLaunchKernelGGL(k_bind_rows<int64_t>, grid, dim3(256), 0, st, (const int64_t *)T, rows, cols, E, per, scratch); break;
    default: hipLaunchKernelGGL(k_bind_rows<uint64_t>, grid, dim3(256), 0, st, (const uint64_t *)T, rows, cols, E, per, scratch); break;
    }
    const ChunkSum cs{scratch, nch, cols, out};
    hipLaunchKernelGGL(k_sum_chunks, dim3(sum_chunks_blocks(cols)), dim3(256), 0, st, cs);
}

ChunkSum launch_bind_rows_chunks(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E,
                                 uint64_t *scratch, uint64_t *out, hipStream_t st)
{
    const int nch = bind_rows_chunks(rows, cols);
    const uint32_t per = (rows + nch - 1) / nch;
    dim3 grid((cols + 63) / 64, nch);
    switch (dtype) {
    case RA_I16: hipLaunchKernelGGL(k_bind_rows<int16_t>, grid, dim3(256), 0, st, (const int16_t *)T, rows, cols, E, per, scratch); break;
    case RA_I32: hipLaunchKernelGGL(k_bind_rows<int32_t>, grid, dim3(256), 0, st, (const int32_t *)T, rows, cols, E, per, scratch); break;
    case RA_I64: hipLaunchKernelGGL(k_bind_rows<int64_t>, grid, dim3(256), 0, st, (const int64_t *)T, rows, cols, E, per, scratch); break;
    default: hipLaunchKernelGGL(k_bind_rows<uint64_t>, grid, dim3(256), 0, st, (const uint64_t *)T, rows, cols, E, per, scratch); break;
    }
    return ChunkSum{scratch, nch, cols, out};
}

// int16 entries, cols >= 8: E[c] = e_hi 2^31 + e_lo (e_lo < 2^31), so
// sum_c E[c] z_c = 2^31 sum e_hi z + sum e_lo z with both sums exact in int64
// (|e z| < 2^46, at most cols / 64 terms per lane): two v_mad_i64_i32 per
// entry and one reduction mod p per lane.  A wave takes four rows and reads
// each eq value once for all of them; lanes take 8 consecutive columns (one
// 16-byte load per row).
constexpr int kBindRowsPerWave = 4;

__global__ __launch_bounds__(256) void k_bind_cols16(const int16_t *__restrict__ B, uint32_t rows, uint32_t cols,
                                                     const uint64_t *__restrict__ E, uint64_t *__restrict__ out,
                                                     uint32_t nmain, ChunkSum cs)
{
    if (blockIdx.x >= nmain) {  // the chunk sums of the other side's binding
        sum_chunks_block(cs, blockIdx.x - nmain);
        return;
    }
    constexpr int RW = kBindRowsPerWave;
    const uint32_t r0 = ((blockIdx.x * blockDim.x + threadIdx.x) >> 6) * RW;  // wave-uniform
    const int lane = threadIdx.x & 63;
    if (r0 >= rows) return;
    int64_t lo[RW], hi[RW];
#pragma unroll
    for (int rr = 0; rr < RW; rr++) lo[rr] = hi[rr] = 0;
    for (uint32_t c0 = 8 * lane; c0 < cols; c0 += 512) {
        int32_t el[8], eh[8];
#pragma unroll
        for (int t = 0; t < 8; t++) {
            const uint64_t e = E[c0 + t];
            el[t] = (int32_t)(e & 0x7FFFFFFFull);
            eh[t] = (int32_t)(e >> 31);
        }
#pragma unroll
        for (int rr = 0; rr < RW; rr++) {
            if (r0 + rr >= rows) break;
            const v4i z4 = *(const v4i *)&B[(size_t)(r0 + rr) * cols + c0];
#pragma unroll
            for (int t = 0; t < 8; t++) {
                const int32_t z = (int32_t)(int16_t)(z4[t >> 1] >> (16 * (t & 1)));
                lo[rr] += (int64_t)el[t] * z;
                hi[rr] += (int64_t)eh[t] * z;
            }
        }
    }
#pragma unroll
    for (int rr = 0; rr < RW; rr++) {
        const uint64_t v = m61::wave_sum(m61::add(m61::from_i64(lo[rr]), m61::rotl(m61::from_i64(hi[rr]), 31)));
        if (lane == 0 && r0 + rr < rows) out[r0 + rr] = v;
    }
}

void launch_bind_cols(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E, uint64_t *out,
                      hipStream_t st, const ChunkSum *cs)
{
    if (dtype == RA_I16 && cols >= 8 && ((uintptr_t)T & 15) == 0) {
        const uint32_t waves = (rows + kBindRowsPerWave - 1) / kBindRowsPerWave, nmain = (waves + 3) / 4;
        const ChunkSum none{nullptr, 0, 0, nullptr};
        const uint32_t extra = cs ? sum_chunks_blocks(cs->cols) : 0;
        hipLaunchKernelGGL(k_bind_cols16, dim3(nmain + extra), dim3(256), 0, st, (const int16_t *)T, rows, cols, E,
                           out, nmain, cs ? *cs : none);
        return;
    }
    if (cs) hipLaunchKernelGGL(k_sum_chunks, dim3(sum_chunks_blocks(cs->cols)), dim3(256), 0, st, *cs);
    dim3 grid((rows + 3) / 4);  // four waves (rows) per block
    switch (dtype) {
    case RA_I16: hipLaunchKernelGGL(k_bind_cols<int16_t>, grid, dim3(256), 0, st, (const int16_t *)T, rows, cols, E, out); break;
    case RA_I32: hipLaunchKernelGGL(k_bind_cols<int32_t>, grid, dim3(256), 0, st, (const int32_t *)T, rows, cols, E, out); break;
    case RA_I64: hipLaunchKernelGGL(k_bind_cols<int64_t>, grid, dim3(256), 0, st, (const int64_t *)T, rows, cols, E, out); break;
    default: hipLaunchKernelGGL(k_bind_cols<uint64_t>, grid, dim3(256), 0, st, (const uint64_t *)T, rows, cols, E, out); break;
    }
}

// ---------------------------------------------------------------------------
// Rescale / ReLU witness (Sec. II-A, Sec. III-A-2, Sec. III-B).
// Pass 1: min and max of C -> t (R is monotone in C, so the extreme R come
// from the extreme C).  Pass 2: R, Rm, Y, Z, the bit word and the four claims.
// ---------------------------------------------------------------------------
int witness_blocks(uint64_t N)
{
    const uint64_t b = (N + kThreads - 1) / kThreads;
    return (int)(b < (uint64_t)kMaxBlocks ? b : (uint64_t)kMaxBlocks);
}

__device__ __forceinline__ int64_t rescale(int64_t c, int s, int mode)
{
    const int64_t half = mode == RA_ROUND_NEAREST ? (int64_t)1 << (s - 1) : 0;
    return (c + half) >> s;  // arithmetic shift = floor division by 2^s
}

// Block min / max of v into (mn, mx) of thread 0.
__device__ __forceinline__ void block_minmax(int64_t &mn, int64_t &mx)
{
    __shared__ int64_t smin[4], smax[4];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const int64_t a = __shfl_xor(mn, off, 64), b = __shfl_xor(mx, off, 64);
        mn = a < mn ? a : mn;
        mx = b > mx ? b : mx;
    }
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    if (lane == 0) {
        smin[wid] = mn;
        smax[wid] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0)
        for (int w = 1; w < (int)(blockDim.x >> 6); w++) {
            mn = smin[w] < mn ? smin[w] : mn;
            mx = smax[w] > mx ? smax[w] : mx;
        }
    __syncthreads();
}

// Pass 1: min and max of C per block, then one block combines them and sets
// t, P and the status.
__global__ __launch_bounds__(256) void k_minmax(const int64_t *__restrict__ C, uint64_t N, int64_t *__restrict__ part)
{
    int64_t mn = INT64_MAX, mx = INT64_MIN;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N; i += (uint64_t)gridDim.x * blockDim.x) {
        const int64_t c = C[i];
        mn = c < mn ? c : mn;
        mx = c > mx ? c : mx;
    }
    block_minmax(mn, mx);
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = mn;
        part[2 * blockIdx.x + 1] = mx;
    }
}

__global__ __launch_bounds__(256) void k_wit_params(const int64_t *__restrict__ part, int nblk, int s, int relu,
                                                    int mode, int t_in, WitParams *__restrict__ prm)
{
    int64_t mn = INT64_MAX, mx = INT64_MIN;
    for (int b = threadIdx.x; b < nblk; b += blockDim.x) {
        mn = part[2 * b] < mn ? part[2 * b] : mn;
        mx = part[2 * b + 1] > mx ? part[2 * b + 1] : mx;
    }
    block_minmax(mn, mx);
    if (threadIdx.x != 0) return;
    WitParams p;
    p.status = 0;
    p.s = s;
    p.relu = relu;
    p.mode = mode;
    p.t_in = t_in;
    p.cmin = mn;
    p.cmax = mx;
    const int64_t rlo = rescale(mn, s, mode), rhi = rescale(mx, s, mode);
    // u = R for R >= 0, -R - 1 for R < 0; R in [-2^(t+1), 2^(t+1)) iff u < 2^(t+1)
    const uint64_t ulo = rlo >= 0 ? (uint64_t)rlo : (uint64_t)(-(rlo + 1));
    const uint64_t uhi = rhi >= 0 ? (uint64_t)rhi : (uint64_t)(-(rhi + 1));
    const uint64_t umax = ulo > uhi ? ulo : uhi;
    int bl = 0;
    while (bl < 64 && (umax >> bl) != 0) bl++;
    int t = bl > 1 ? bl - 1 : 0;
    if (t_in >= 0) {
        if (t_in < 62 && (umax >> (t_in + 1)) != 0) p.status = RA_E_RANGE;
        t = t_in;
    }
    if (p.status == 0 && s + t + 3 > 61) p.status = RA_E_FIELD_TOO_SMALL;
    if (p.status == 0 && t > 29) p.status = RA_E_NOT_IMPLEMENTED;  // R, Y must fit int32
    const int Q = s + (t + 2) * (relu ? 2 : 1);
    int P = 1, lP = 0;
    while (P < Q) {
        P <<= 1;
        lP++;
    }
    if (p.status == 0 && lP > kMaxPlaneLog) p.status = RA_E_NOT_IMPLEMENTED;  // one bit word per output
    p.t = t;
    p.P = P;
    p.lP = lP;
    *prm = p;
}

// Pass 2: R, Rm, Y, Z, the bit word and per-block claims, then one block
// sums the claims (R~, Rm~, Y~, Z~ at (r1, r2)) and mirrors the parameters and
// claims to `mirror` (12 words) when it is given.
// With t given (known != 0) the parameters come by value and every workgroup
// also flags, in flags[block], whether one of its R lies outside the range;
// the final kernel turns the flags into the status.
// Blocks of the rescale pass: V = 4 outputs per thread, one pass over N for
// up to kMaxBlocks blocks (never more blocks than witness_blocks(N)).
static int rescale_blocks(uint64_t N)
{
    const uint64_t b = (N + 4 * kThreads - 1) / (4 * kThreads);
    return (int)(b < (uint64_t)kMaxBlocks ? b : (uint64_t)kMaxBlocks);
}

// Pass 2: R, Rm, Y, Z, the bit word and per-block claims, then one block
// sums the claims (R~, Rm~, Y~, Z~ at (r1, r2)) and mirrors the parameters and
// claims to `mirror` (12 words) when it is given.
// With t given (known != 0) the parameters come by value and every workgroup
// also flags, in flags[block], whether one of its R lies outside the range;
// the final kernel turns the flags into the status.
// A thread takes V consecutive outputs per step (V = 4: 16-byte loads and
// stores; V = 1 for N < 4 or unaligned buffers).
template <int V>
__global__ __launch_bounds__(256) void k_rescale(const int64_t *__restrict__ C, uint64_t N, int lk,
                                                 const WitParams *__restrict__ prm, const uint64_t *__restrict__ E1,
                                                 const uint64_t *__restrict__ E2, int32_t *__restrict__ R,
                                                 uint16_t *__restrict__ Rm, int32_t *__restrict__ Y,
                                                 int32_t *__restrict__ Z, uint64_t *__restrict__ bits,
                                                 uint64_t *__restrict__ claim_part, WitParams hp, int known,
                                                 uint32_t *__restrict__ flags)
{
    typedef long long v2l __attribute__((ext_vector_type(2)));
    typedef int v4i_t __attribute__((ext_vector_type(4)));
    typedef unsigned short v4u16 __attribute__((ext_vector_type(4)));
    __shared__ uint64_t red[m61::block_sum_words(4, 256)];
    const WitParams p = known ? hp : *prm;
    if (p.status != 0) return;  // uniform over the grid
    const int s = p.s, t = p.t, relu = p.relu;
    const int64_t half = p.mode == RA_ROUND_NEAREST ? (int64_t)1 << (s - 1) : 0;
    const uint64_t kmask = (1ull << lk) - 1;
    uint64_t acc[4] = {0, 0, 0, 0};
    int out_of_range = 0;
    const uint64_t ng = N / V;
    for (uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; g < ng; g += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t x0 = g * V;
        int64_t c[V];
        uint64_t el[V], eh[V];
        if constexpr (V == 4) {
            const v2l c01 = *(const v2l *)&C[x0], c23 = *(const v2l *)&C[x0 + 2];
            c[0] = c01[0];
            c[1] = c01[1];
            c[2] = c23[0];
            c[3] = c23[1];
        } else {
            c[0] = C[x0];
        }
#pragma unroll
        for (int i = 0; i < V; i++) {
            const uint64_t x = x0 + i;
            const uint64_t e = m61::lmul(E1[x >> lk], E2[x & kmask]);
            el[i] = e & 0x7FFFFFFFull;
            eh[i] = e >> 31;
        }
        int32_t r[V], rm[V], y[V], z[V];
        uint64_t w[V];
#pragma unroll
        for (int i = 0; i < V; i++) {
            const WitOut o = witness_entry(c[i], s, t, relu, half, out_of_range);
            r[i] = o.r;
            rm[i] = o.rm;
            y[i] = o.y;
            z[i] = o.z;
            w[i] = o.w;
        }
        if constexpr (V == 4) {
            *(v4i_t *)&R[x0] = v4i_t{r[0], r[1], r[2], r[3]};
            *(v4i_t *)&Y[x0] = v4i_t{y[0], y[1], y[2], y[3]};
            *(v4i_t *)&Z[x0] = v4i_t{z[0], z[1], z[2], z[3]};
            *(v4u16 *)&Rm[x0] = v4u16{(unsigned short)rm[0], (unsigned short)rm[1], (unsigned short)rm[2],
                                      (unsigned short)rm[3]};
            *(v2l *)&bits[x0] = v2l{(long long)w[0], (long long)w[1]};
            *(v2l *)&bits[x0 + 2] = v2l{(long long)w[2], (long long)w[3]};
        } else {
            R[x0] = r[0];
            Y[x0] = y[0];
            Z[x0] = z[0];
            Rm[x0] = (uint16_t)rm[0];
            bits[x0] = w[0];
        }
        acc[0] = m61::fold(acc[0] + claim_terms<V>(el, eh, r));
        acc[1] = m61::fold(acc[1] + claim_terms<V>(el, eh, rm));
        acc[2] = m61::fold(acc[2] + claim_terms<V>(el, eh, y));
        acc[3] = m61::fold(acc[3] + claim_terms<V>(el, eh, z));
    }
    if (known) {
        const int any = __syncthreads_or(out_of_range);
        if (threadIdx.x == 0) flags[blockIdx.x] = (uint32_t)any;
    }
    m61::block_sum<4>(acc, red);
    if (threadIdx.x == 0)
        for (int i = 0; i < 4; i++) claim_part[4 * blockIdx.x + i] = acc[i];
}

__global__ __launch_bounds__(256) void k_claims_final(ClaimsJob j)
{
    __shared__ uint64_t red[m61::block_sum_words(4, 256)];
    claims_final_block(j, red, nullptr);
}

void launch_claims_final(const ClaimsJob &j, hipStream_t st)
{
    hipLaunchKernelGGL(k_claims_final, dim3(1), dim3(kThreads), 0, st, j);
}

void launch_witness_params(const int64_t *C, uint64_t N, int s, int relu, int mode, int t_in, int64_t *mm_part,
                           WitParams *params, hipStream_t st)
{
    const int nb = witness_blocks(N);
    hipLaunchKernelGGL(k_minmax, dim3(nb), dim3(kThreads), 0, st, C, N, mm_part);
    hipLaunchKernelGGL(k_wit_params, dim3(1), dim3(256), 0, st, (const int64_t *)mm_part, nb, s, relu, mode, t_in,
                       params);
}

void launch_witness_rescale(const int64_t *C, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2, int32_t *R,
                            uint16_t *Rm, int32_t *Y, int32_t *Z, uint64_t *bits, uint64_t *claim_part,
                            WitParams *params, uint64_t *claims_out, uint64_t *mirror, hipStream_t st,
                            const WitParams *known, uint32_t *flags, ClaimsJob *defer)
{
    const WitParams hp = known ? *known : WitParams{};
    const bool vec = N >= 4 && (((uintptr_t)C | (uintptr_t)R | (uintptr_t)Y | (uintptr_t)Z | (uintptr_t)bits) & 15) == 0 &&
                     ((uintptr_t)Rm & 7) == 0;
    const int nb = vec ? rescale_blocks(N) : witness_blocks(N);
    if (vec)
        hipLaunchKernelGGL(k_rescale<4>, dim3(nb), dim3(kThreads), 0, st, C, N, lk, (const WitParams *)params, E1, E2,
                           R, Rm, Y, Z, bits, claim_part, hp, known ? 1 : 0, flags);
    else
        hipLaunchKernelGGL(k_rescale<1>, dim3(nb), dim3(kThreads), 0, st, C, N, lk, (const WitParams *)params, E1, E2,
                           R, Rm, Y, Z, bits, claim_part, hp, known ? 1 : 0, flags);
    const ClaimsJob j{claim_part, nb, params, claims_out, mirror, hp, known ? 1 : 0, flags};
    if (defer) *defer = j;
    else launch_claims_final(j, st);
}

}  // namespace ra
