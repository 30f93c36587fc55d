// gemm.hip -- the exact integer product C = A B (Alg. 1 step 2) on the
// matrix cores.
//
// Every entry is split into signed 8-bit limbs of an offset value:
//   b = 256 b1 + b0 + 128                  (b0 = (b & 255) - 128, b1 = b >> 8),
//   a = sum_u 256^u a_u + c_A              (LA = 2 limbs for int16, 4 for int32;
//                                            lower limbs shifted by -128, c_A the sum of the shifts),
// so with A~ = sum_u 256^u A_u and B~ = 256 B1 + B0 (entries a - c_A, b - 128)
//   A B = A~ B~ + 128 rowsum(A)_i + c_A colsum(B)_j - 128 c_A m,
//   A~ B~ = sum_w 256^w S_w,  S_w = sum_{u + v = w} A_u B_v.
// Each S_w is an int8 x int8 -> int32 matrix product (v_mfma_i32_32x32x32_i8);
// at most two limb products share a weight, so |S_w| <= 2 m 2^14 fits int32
// for m <= 32768, and the int64 recombination is exact.
#include "common.hpp"
#include "claims.hpp"
#include "tail.hpp"

namespace ra {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kTile = 64;    // block tile (rows and columns)
// LDS stages (k steps of 64) per block: 48 KB for int16 A (three blocks fit
// a CU, so the matrix tail's workgroup runs beside two tiles per CU), 72 KB
// for int32 A.  A fourth stage for int16 A was slower.
template <int LA> constexpr int gemm_stages() { return 3; }

__host__ __device__ inline uint32_t round_up64(uint32_t v) { return (v + 63u) & ~63u; }

// Limb planes are stored as MFMA fragments.  For a block of 32 rows R and a
// block of 32 bytes q along the inner dimension, the 64 lanes' 16-byte
// operands of v_mfma_i32_32x32x32_i8 (lane l: row 32 R + (l & 31), bytes
// 32 q + 16 (l >> 5) .. + 16) lie contiguously in 1 KB, at
// frag_off(plane, R, q) + 16 l, so one wave moves a whole fragment with one
// 16-byte load per lane.
__host__ __device__ inline size_t frag_off(int plane, uint32_t R, uint32_t q, uint32_t nR, uint32_t nQ)
{
    return (((size_t)plane * nR + R) * nQ + q) * 1024;
}
__host__ __device__ inline uint32_t frag_lane(uint32_t row, uint32_t kb) { return (row & 31) + 32 * ((kb >> 4) & 1); }

typedef __attribute__((address_space(3))) int8_t lds_i8;

// Wait until at most N of the wave's LDS reads are outstanding; the operands
// of the half that has then landed pass through the wait, so that nothing
// that uses them is scheduled before it.  (Each step's operands are fresh
// values, so no register copy of them can precede the wait.)
template <int N, int LA>
__device__ __forceinline__ void lds_wait(v4i (&a)[LA], v4i (&b)[2])
{
    static_assert(N >= 0 && N < 16, "lgkmcnt field");
    static_assert(LA >= 2 && LA <= 4, "limbs of A");
    if constexpr (LA == 2)
        asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]) : "i"(N) : "memory");
    else if constexpr (LA == 3)
        asm volatile("s_waitcnt lgkmcnt(%5)"
                     : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(b[0]), "+v"(b[1])
                     : "i"(N)
                     : "memory");
    else
        asm volatile("s_waitcnt lgkmcnt(%6)"
                     : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1])
                     : "i"(N)
                     : "memory");
}

// s_waitcnt that waits until at most N vector-memory operations of the wave
// are outstanding (expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void vm_wait()
{
    static_assert(N >= 0 && N < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Byte gathers: v_perm_b32 picks bytes of {hi, lo} (selector bytes 0-3 from
// lo, 4-7 from hi, 0x0c gives zero).
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// A (n x m) -> limb planes Al[u][np][mp] (zero padded) and rowsum(A).  One
// wave per row; a lane takes 16 consecutive entries and writes 16 bytes per
// limb: the lower limbs shifted by -128 (a xor of the sign bit), the top limb
// as is.  For int32, rowlimb[row] = 3 when the row's top plane is all zero
// (every entry in [0, 2^24), as the ReLU outputs of a layer are), else 4: a
// product tile whose rows all have three limbs skips plane 3.
template <typename TA, int LA>
__device__ __forceinline__ void split_a_block(const TA *__restrict__ A, uint32_t n, uint32_t m, uint32_t np,
                                              uint32_t mp, int8_t *__restrict__ Al, int64_t *__restrict__ rowsum,
                                              int32_t *__restrict__ rowlimb, uint32_t blk)
{
    const uint32_t row = blk * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= np) return;  // wave-uniform
    uint32_t top = 0;       // OR of the top plane's words
    int64_t s = 0;
    for (uint32_t c = lane * 16; c < mp; c += 1024) {
        v4i out[LA];
        if (row < n && c < m && c + 16 > m) {  // partial chunk (m < 16): entry by entry, padding zero
#pragma unroll
            for (int w = 0; w < 4; w++) {
                uint32_t wd[LA];
#pragma unroll
                for (int u = 0; u < LA; u++) wd[u] = 0;
#pragma unroll
                for (int b = 0; b < 4; b++) {
                    const uint32_t l = c + 4 * w + b;
                    if (l >= m) continue;
                    const int32_t a = (int32_t)A[(size_t)row * m + l];
                    s += a;
#pragma unroll
                    for (int u = 0; u < LA; u++) {
                        const int32_t d = u == LA - 1 ? (a >> (8 * u)) : (((a >> (8 * u)) & 255) - 128);
                        wd[u] |= (uint32_t)(uint8_t)(int8_t)d << (8 * b);
                    }
                }
#pragma unroll
                for (int u = 0; u < LA; u++) out[u][w] = (int)wd[u];
            }
        } else if (row < n && c < m) {  // whole 16-entry chunk
            constexpr int NV = sizeof(TA) * 16 / 16;
            v4i in[NV];
#pragma unroll
            for (int q = 0; q < NV; q++) in[q] = *(const v4i *)&A[(size_t)row * m + c + q * (16 / sizeof(TA))];
            if (sizeof(TA) == 2) {
#pragma unroll
                for (int w = 0; w < 4; w++) {  // entries 4w .. 4w+3 in dwords 2w, 2w+1
                    const uint32_t d0 = (uint32_t)in[w >> 1][2 * (w & 1)], d1 = (uint32_t)in[w >> 1][2 * (w & 1) + 1];
                    out[0][w] = (int)(perm(d1, d0, 0x06040200u) ^ 0x80808080u);
                    out[LA - 1][w] = (int)perm(d1, d0, 0x07050301u);
                    s += (int32_t)(int16_t)d0 + (int32_t)(int16_t)(d0 >> 16) + (int32_t)(int16_t)d1 +
                         (int32_t)(int16_t)(d1 >> 16);
                }
            } else {
#pragma unroll
                for (int w = 0; w < 4; w++) {  // entries 4w .. 4w+3 are in[w][0..3]
                    const uint32_t d0 = in[w][0], d1 = in[w][1], d2 = in[w][2], d3 = in[w][3];
#pragma unroll
                    for (int u = 0; u < LA; u++) {
                        const uint32_t lo = perm(d1, d0, 0x0c0c0000u | ((4 + u) << 8) | u);
                        const uint32_t hi = perm(d3, d2, (((4 + u) << 24) | (u << 16)) | 0x0c0cu);
                        out[u][w] = (int)((lo | hi) ^ (u < LA - 1 ? 0x80808080u : 0u));
                    }
                    s += (int64_t)(int32_t)d0 + (int32_t)d1 + (int32_t)d2 + (int32_t)d3;
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < LA; u++) out[u] = v4i{0, 0, 0, 0};
        }
        top |= (uint32_t)(out[LA - 1][0] | out[LA - 1][1] | out[LA - 1][2] | out[LA - 1][3]);
#pragma unroll
        for (int u = 0; u < LA; u++)
            *(v4i *)&Al[frag_off(u, row >> 5, c >> 5, np >> 5, mp >> 5) + 16 * frag_lane(row, c)] = out[u];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0 && row < n) rowsum[row] = s;
    if (LA == 4) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) top |= (uint32_t)__shfl_xor((int)top, off, 64);
        if (lane == 0) rowlimb[row] = top ? 4 : 3;
    }
}

// B (m x k) -> transposed limb planes Bt[v][kp][mp] (row j holds column j of
// B, zero padded) and the column sums of every 64-row tile, colpart[ti][j].
// The 64 x 64 tile goes through LDS; four threads take one column's 64 bytes
// (16 each), so a wave writes whole 64-byte segments.
__device__ __forceinline__ void split_bt_block(const int16_t *__restrict__ B, uint32_t m, uint32_t k, uint32_t mp,
                                               uint32_t kp, int8_t *__restrict__ Bt, int64_t *__restrict__ colpart,
                                               uint32_t bx, uint32_t by)
{
    __shared__ int16_t t[64][66];
    __shared__ int32_t cs[4][64];
    const uint32_t l0 = by * 64, j0 = bx * 64;
    const int tid = threadIdx.x;
    {   // load: thread -> row tid / 4, 16 consecutive columns
        const int r = tid >> 2, c = (tid & 3) * 16;
        const uint32_t l = l0 + r;
        if (l < m && j0 + c + 16 <= k && (k & 7) == 0) {  // two aligned 16-byte reads
            const v4i v0 = *(const v4i *)&B[(size_t)l * k + j0 + c], v1 = *(const v4i *)&B[(size_t)l * k + j0 + c + 8];
#pragma unroll
            for (int e = 0; e < 4; e++) {
                *(int32_t *)&t[r][c + 2 * e] = v0[e];
                *(int32_t *)&t[r][c + 8 + 2 * e] = v1[e];
            }
        } else {
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const uint32_t j = j0 + c + e;
                t[r][c + e] = (l < m && j < k) ? B[(size_t)l * k + j] : (int16_t)0;
            }
        }
    }
    __syncthreads();
    const int jj = tid >> 2, ch = (tid & 3) * 16;
    const uint32_t j = j0 + jj;
    v4i o0, o1;
    int32_t sum = 0;
#pragma unroll
    for (int w = 0; w < 4; w++) {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int b = 0; b < 4; b++) {
            const int lr = ch + 4 * w + b;
            const int32_t v = t[lr][jj];
            const bool in = l0 + lr < m && j < k;
            sum += v;
            lo |= (uint32_t)(uint8_t)(in ? (int8_t)((v & 255) - 128) : (int8_t)0) << (8 * b);
            hi |= (uint32_t)(uint8_t)(in ? (int8_t)(v >> 8) : (int8_t)0) << (8 * b);
        }
        o0[w] = (int)lo;
        o1[w] = (int)hi;
    }
    const uint32_t kb = l0 + ch;
    *(v4i *)&Bt[frag_off(0, j >> 5, kb >> 5, kp >> 5, mp >> 5) + 16 * frag_lane(j, kb)] = o0;
    *(v4i *)&Bt[frag_off(1, j >> 5, kb >> 5, kp >> 5, mp >> 5) + 16 * frag_lane(j, kb)] = o1;
    cs[tid & 3][jj] = sum;
    __syncthreads();
    if (tid < 64 && j0 + tid < k)
        colpart[(size_t)by * kp + j0 + tid] = (int64_t)cs[0][tid] + cs[1][tid] + cs[2][tid] + cs[3][tid];
}

// Both operands in one launch: workgroups below na split rows of A (four per
// workgroup), the others 64 x 64 tiles of B.
template <typename TA, int LA>
__global__ __launch_bounds__(256) void k_split(const TA *__restrict__ A, uint32_t n, uint32_t m, uint32_t np,
                                               uint32_t mp, int8_t *__restrict__ Al, int64_t *__restrict__ rowsum,
                                               int32_t *__restrict__ rowlimb, uint32_t na,
                                               const int16_t *__restrict__ B, uint32_t k, uint32_t kp,
                                               int8_t *__restrict__ Bt, int64_t *__restrict__ colpart)
{
    if (blockIdx.x < na) {
        split_a_block<TA, LA>(A, n, m, np, mp, Al, rowsum, rowlimb, blockIdx.x);
        return;
    }
    const uint32_t t = blockIdx.x - na, tx = kp / 64;
    split_bt_block(B, m, k, mp, kp, Bt, colpart, t % tx, t / tx);
}

// ---------------------------------------------------------------------------
// The front of the matrix call in one launch.  Every role reads only the
// operands A, B and the challenge point (r1, r2), so they run side by side:
//   - the limb split of A and B for the exact product (above);
//   - the row binding a(l) = sum_i eq(r1, i) A[i, l] and the column binding
//     b(l) = sum_j B[l, j] eq(r2, j) of Eq. (4);
//   - the eq tables E1 = eq(r1, .), E2 = eq(r2, .) for the later calls.
// The binding roles build eq values from two small factor tables in LDS:
// with lb = v / 2 low variables, eq(z, i) = H[i >> lb] L[i mod 2^lb], where H
// is the eq vector of the first v - lb coordinates of z and L that of the
// last lb (Eq. (1) factors over the coordinates).
// ---------------------------------------------------------------------------
constexpr int kFrontMaxLog = 16;   // largest log n, log k of the fused front (factor tables <= 256 words)

// H (2^(v - v/2) words) and L (2^(v/2) words) for the point z (v <= 16);
// folded values.  The point is staged in LDS first (zs, kFrontMaxLog words),
// so the products wait on one load, not one per coordinate.  The caller
// synchronises.
__device__ __forceinline__ void eq_factors(const uint64_t *__restrict__ z, int v, uint64_t *H, uint64_t *L,
                                           uint64_t *zs)
{
    if ((int)threadIdx.x < v) zs[threadIdx.x] = z[threadIdx.x];
    __syncthreads();
    const int lb = v / 2, hb = v - lb, nh = 1 << hb;
    for (int i = threadIdx.x; i < nh + (1 << lb); i += blockDim.x) {
        const bool high = i < nh;
        const int idx = high ? i : i - nh, nv = high ? hb : lb, j0 = high ? 0 : hb;
        uint64_t acc = 1;
        for (int j = 0; j < nv; j++) {
            const uint64_t zj = zs[j0 + j];
            acc = m61::lmul(acc, ((idx >> (nv - 1 - j)) & 1) ? zj : m61::lsub(1, zj));
        }
        (high ? H : L)[idx] = acc;
    }
}

// Row binding of one chunk of rows for 64 columns.  A lane takes 16 bytes
// (CPL entries) of a row per step; G lanes cover the 64 columns and RS row
// slots interleave.  Each eq value e (< 2^62) is cut into NL limbs of LB bits,
// so sum_i e_i z_i is accumulated exactly in int64 per limb (|limb z| < 2^46
// for int16, < 2^52 for int32, at most 2^11 rows per lane), then reduced
// mod p once.  The chunk's canonical sums are added to acc (low 32 bits at
// acc[c], the rest at acc[m + c]), which the first reader of a turns into
// field values and clears.
template <typename T>
__device__ __forceinline__ void front_rowbind(const T *__restrict__ A, uint32_t n, uint32_t m, const uint64_t *r1,
                                              int ln, uint32_t rpc, uint32_t blk, uint64_t *acc, uint64_t *tab,
                                              uint64_t *red)
{
    constexpr int CPL = 16 / (int)sizeof(T), G = 64 / CPL, RS = 256 / G;
    constexpr int NL = sizeof(T) == 2 ? 2 : 3, LB = sizeof(T) == 2 ? 31 : 21;
    constexpr uint64_t LMASK = (1ull << LB) - 1;
    uint64_t *H = tab, *Lt = tab + 256;
    eq_factors(r1, ln, H, Lt, tab + 512);
    __syncthreads();
    const uint32_t ncb = m / 64, cb = blk % ncb, ch = blk / ncb;
    const int tid = threadIdx.x, g = tid % G, slot = tid / G;
    const uint32_t c = cb * 64 + g * CPL, r0 = ch * rpc, re = r0 + rpc < n ? r0 + rpc : n;
    const int lb = ln / 2;
    const uint32_t lmask = (1u << lb) - 1;
    int64_t s[CPL][NL];
#pragma unroll
    for (int q = 0; q < CPL; q++)
#pragma unroll
        for (int l = 0; l < NL; l++) s[q][l] = 0;
    for (uint32_t rb = r0 + slot; rb < re; rb += 4 * RS) {
        v4i z4[4];
        uint64_t e[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {  // loads first
            const uint32_t r = rb + u * RS;
            z4[u] = r < re ? *(const v4i *)&A[(size_t)r * m + c] : v4i{0, 0, 0, 0};
            e[u] = r < re ? m61::lmul(H[r >> lb], Lt[r & lmask]) : 0;
        }
#pragma unroll
        for (int u = 0; u < 4; u++) {
            int64_t el[NL];
#pragma unroll
            for (int l = 0; l < NL; l++) el[l] = (int64_t)(l == NL - 1 ? e[u] >> (LB * l) : (e[u] >> (LB * l)) & LMASK);
#pragma unroll
            for (int q = 0; q < CPL; q++) {
                const int32_t z = sizeof(T) == 2 ? (int32_t)(int16_t)(z4[u][q >> 1] >> (16 * (q & 1))) : z4[u][q];
#pragma unroll
                for (int l = 0; l < NL; l++) s[q][l] += el[l] * z;
            }
        }
    }
#pragma unroll
    for (int q = 0; q < CPL; q++) {
        uint64_t v = 0;
#pragma unroll
        for (int l = 0; l < NL; l++) v = m61::add(v, m61::rotl(m61::from_i64(s[q][l]), LB * l));
        red[slot * 65 + g * CPL + q] = v;
    }
    __syncthreads();
    if (tid < 64) {
        uint64_t v = 0;
#pragma unroll 4
        for (int u = 0; u < RS; u++) v = m61::fold(v + red[u * 65 + tid]);
        v = m61::canon(v);
        atomicAdd((unsigned long long *)&acc[cb * 64 + tid], (unsigned long long)(v & 0xFFFFFFFFull));
        atomicAdd((unsigned long long *)&acc[m + cb * 64 + tid], (unsigned long long)(v >> 32));
    }
}

// Column binding of RW rows per wave (4 RW per workgroup): lanes take 8
// consecutive columns per step (one 16-byte load per row); eq(r2, c) =
// e_hi 2^31 + e_lo is accumulated exactly per half in int64, one reduction
// mod p per lane and row.  Four rows per wave share each eq value; one row
// per wave gives small matrices four times the workgroups (more waves in
// flight for a latency-bound role).
template <int RW>
__device__ __forceinline__ void front_colbind(const int16_t *__restrict__ B, uint32_t rows, uint32_t cols,
                                              const uint64_t *r2, int lk, uint32_t blk, uint64_t *out, uint64_t *tab)
{
    uint64_t *H = tab, *Lt = tab + 256;
    eq_factors(r2, lk, H, Lt, tab + 512);
    __syncthreads();
    const int lb = lk / 2;
    const uint32_t lmask = (1u << lb) - 1;
    const uint32_t r0 = blk * 4 * RW + (threadIdx.x >> 6) * RW;  // wave-uniform
    const int lane = threadIdx.x & 63;
    if (r0 >= rows) return;
    int64_t lo[RW], hi[RW];
#pragma unroll
    for (int rr = 0; rr < RW; rr++) lo[rr] = hi[rr] = 0;
    for (uint32_t c0 = 8 * lane; c0 < cols; c0 += 512) {
        v4i z4[RW];
#pragma unroll
        for (int rr = 0; rr < RW; rr++)
            z4[rr] = r0 + rr < rows ? *(const v4i *)&B[(size_t)(r0 + rr) * cols + c0] : v4i{0, 0, 0, 0};
        int32_t el[8], eh[8];
#pragma unroll
        for (int t = 0; t < 8; t++) {
            const uint32_t cc = c0 + t;
            const uint64_t e = m61::lmul(H[cc >> lb], Lt[cc & lmask]);  // < 2^61 + 8
            el[t] = (int32_t)(e & 0x7FFFFFFFull);
            eh[t] = (int32_t)(e >> 31);
        }
#pragma unroll
        for (int rr = 0; rr < RW; rr++)
#pragma unroll
            for (int t = 0; t < 8; t++) {
                const int32_t z = (int32_t)(int16_t)(z4[rr][t >> 1] >> (16 * (t & 1)));
                lo[rr] += (int64_t)el[t] * z;
                hi[rr] += (int64_t)eh[t] * z;
            }
    }
#pragma unroll
    for (int rr = 0; rr < RW; rr++) {
        const uint64_t v = m61::wave_sum(m61::add(m61::from_i64(lo[rr]), m61::rotl(m61::from_i64(hi[rr]), 31)));
        if (lane == 0 && r0 + rr < rows) out[r0 + rr] = v;
    }
}

// 1024 entries of eq(z, .) (v <= 16 variables), canonical.
__device__ __forceinline__ void front_eq(const uint64_t *z, int v, uint64_t *out, uint32_t blk, uint64_t *tab)
{
    uint64_t *H = tab, *Lt = tab + 256;
    eq_factors(z, v, H, Lt, tab + 512);
    __syncthreads();
    const int lb = v / 2;
    const uint32_t lmask = (1u << lb) - 1, nv = 1u << v;
#pragma unroll
    for (int u = 0; u < 4; u++) {
        const uint32_t i = blk * 1024 + u * 256 + threadIdx.x;
        if (i < nv) out[i] = m61::canon(m61::lmul(H[i >> lb], Lt[i & lmask]));
    }
}

struct FrontArgs {
    const void *A;
    const int16_t *B;
    uint32_t n, m, k, np, mp, kp;
    int8_t *Al;
    int64_t *rowsum;
    int32_t *rowlimb;
    int8_t *Bt;
    int64_t *colpart;
    const uint64_t *r1, *r2;
    int ln, lk;
    uint64_t *acc;       // row binding accumulators (2 m words, zero on entry)
    uint64_t *b;         // column binding (m words)
    uint64_t *E1, *E2;   // eq tables for the later calls
    uint32_t rpc;        // rows per row-binding chunk
    uint32_t n_rb, n_cb, n_sb, n_sa, n_e1;  // workgroups per role (the E2 table's follow E1's)
};

template <typename TA, int LA, int RW>
__global__ __launch_bounds__(256) void k_front(FrontArgs f)
{
    __shared__ uint64_t tab[512 + kFrontMaxLog];  // eq factors H, L and the point
    __shared__ uint64_t red[(256 / (64 / (16 / (int)sizeof(TA)))) * 65];
    uint32_t b = blockIdx.x;
    // The four heavy roles, then the eq tables.  Workgroups start in index
    // order, so the roles whose workgroups run longest go first and the short
    // tiles of the split of B fill in behind them: with four rows per
    // column-binding wave (large m, RW = 4) that role has the longest loop,
    // then the split of A (a whole row per wave); with one row per wave the
    // row binding leads and the split of A trails.
    if constexpr (RW == 4) {
        if (b < f.n_cb) {
            front_colbind<RW>(f.B, f.m, f.k, f.r2, f.lk, b, f.b, tab);
            return;
        }
        b -= f.n_cb;
        if (b < f.n_sa) {
            split_a_block<TA, LA>((const TA *)f.A, f.n, f.m, f.np, f.mp, f.Al, f.rowsum, f.rowlimb, b);
            return;
        }
        b -= f.n_sa;
        if (b < f.n_rb) {
            front_rowbind<TA>((const TA *)f.A, f.n, f.m, f.r1, f.ln, f.rpc, b, f.acc, tab, red);
            return;
        }
        b -= f.n_rb;
        if (b < f.n_sb) {
            split_bt_block(f.B, f.m, f.k, f.mp, f.kp, f.Bt, f.colpart, b % (f.kp / 64), b / (f.kp / 64));
            return;
        }
        b -= f.n_sb;
    } else {
        if (b < f.n_rb) {
            front_rowbind<TA>((const TA *)f.A, f.n, f.m, f.r1, f.ln, f.rpc, b, f.acc, tab, red);
            return;
        }
        b -= f.n_rb;
        if (b < f.n_cb) {
            front_colbind<RW>(f.B, f.m, f.k, f.r2, f.lk, b, f.b, tab);
            return;
        }
        b -= f.n_cb;
        if (b < f.n_sb) {
            split_bt_block(f.B, f.m, f.k, f.mp, f.kp, f.Bt, f.colpart, b % (f.kp / 64), b / (f.kp / 64));
            return;
        }
        b -= f.n_sb;
        if (b < f.n_sa) {
            split_a_block<TA, LA>((const TA *)f.A, f.n, f.m, f.np, f.mp, f.Al, f.rowsum, f.rowlimb, b);
            return;
        }
        b -= f.n_sa;
    }
    if (b < f.n_e1) front_eq(f.r1, f.ln, f.E1, b, tab);
    else front_eq(f.r2, f.lk, f.E2, b - f.n_e1, tab);
}

// The k loop of one 64 x 64 tile: LE limb planes of A (LE <= LA; planes past
// LE are zero for every row of the tile) and two of B.  Every step needs
// F = 2 (2 LE + 4) fragments (two 32-byte halves of A: LE limbs x 2 row
// blocks, and of B: 2 limbs x 2 column blocks), F / 4 per wave, fetched
// straight into LDS (global_load_lds_dwordx4) S - 1 steps ahead.
template <int LA, int LE, int S>
__device__ __forceinline__ void gemm_loop(const int8_t *__restrict__ Al, const int8_t *__restrict__ Bt, uint32_t bi,
                                          uint32_t bj, uint32_t nR, uint32_t nC, uint32_t nQ, uint32_t nS,
                                          int8_t *stage0, v16i (&acc)[LA == 2 ? 4 : LA + 1])
{
    constexpr int F1 = 2 * LE + 4, F = 2 * F1, FW = F / 4;
    static_assert(F % 4 == 0, "fragments per wave");
    static_assert(S >= 2, "a stage read while the next fills");
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wr = wv >> 1, wc = wv & 1;
    const int8_t *src[FW];
#pragma unroll
    for (int e = 0; e < FW; e++) {
        const int f = FW * wv + e, kk = f / F1, f1 = f % F1;
        src[e] = (f1 < 2 * LE ? Al + frag_off(f1 >> 1, 2 * bi + (f1 & 1), kk, nR, nQ)
                              : Bt + frag_off((f1 - 2 * LE) >> 1, 2 * bj + ((f1 - 2 * LE) & 1), kk, nC, nQ)) +
                 16 * lane;
    }
    auto issue1 = [&](uint32_t q, int sl, int e) {
        __builtin_amdgcn_global_load_lds((const void *)(src[e] + (size_t)q * 2048),
                                         (__attribute__((address_space(3))) void *)(stage0 +
                                                                                    ((size_t)sl * F + FW * wv + e) * 1024),
                                         16, 0, 0);
    };
    auto issue = [&](uint32_t q, int sl) {
#pragma unroll
        for (int e = 0; e < FW; e++) issue1(q, sl, e);
    };
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_i8 *)stage0 + 16 * lane;
#pragma unroll
    for (int q = 0; q < S - 1; q++)
        if ((uint32_t)q < nS) issue(q, q);
    for (uint32_t q = 0; q < nS; q++) {
        // this wave's fragments of step q have landed once at most (S - 2) later
        // steps are in flight
        if (q + S - 2 < nS) vm_wait<(S - 2) * FW>();
        else vm_wait<0>();
        // every wave's fragments of step q have landed, and every wave is done
        // with step q - 1 (a plain barrier: a fence here would also wait for
        // the steps still in flight)
        asm volatile("s_barrier" ::: "memory");
        // Step q + S - 1's fetches go out one at a time between this step's
        // MFMAs (below): issued together after the barrier, a wave waits until
        // the fetch path has taken them all before its first MFMA, and the
        // fetch path then idles while the MFMAs run (timing copies: 1190 ->
        // 770 cycles per step for int16 A, 1396 -> 1021 for int32 A).
        const bool more = q + S - 1 < nS;
        const uint32_t qn = q + S - 1;
        const int sn = (int)(qn % S);
        // The operands are read with explicit LDS reads: the compiler cannot
        // tell which stage a pending LDS DMA writes and would otherwise wait
        // for all of them before any LDS read.  The second 32-byte half is
        // still being read while the first half's MFMAs run.
        const uint32_t sa = lds0 + (q % S) * (F * 1024) + 1024 * wr, sb = sa + 1024 * (wc - wr);
        v4i a[2][LE], b[2][2];
#pragma unroll
        for (int kk = 0; kk < 2; kk++) {
#pragma unroll
            for (int u = 0; u < LE; u++)
                asm volatile("ds_read_b128 %0, %1 offset:%2"
                             : "=v"(a[kk][u])
                             : "v"(sa), "i"((kk * F1 + 2 * u) * 1024)
                             : "memory");
#pragma unroll
            for (int v = 0; v < 2; v++)
                asm volatile("ds_read_b128 %0, %1 offset:%2"
                             : "=v"(b[kk][v])
                             : "v"(sb), "i"((kk * F1 + 2 * LE + 2 * v) * 1024)
                             : "memory");
        }
#pragma unroll
        for (int kk = 0; kk < 2; kk++) {
            if (kk == 0) lds_wait<LE + 2, LE>(a[0], b[0]);
            else lds_wait<0, LE>(a[1], b[1]);
            // limb pairs (u, v) in an order that puts at least two other MFMAs
            // between two updates of one accumulator: int16 A has one
            // accumulator per pair (2 u + v), int32 A one per weight u + v
#pragma unroll
            for (int i = 0; i < 2 * LE; i++) {
                const int u = LE == 3 ? (i < 3 ? i : i == 3 ? 2 : i - 4) : i % LE;
                const int v = LE == 3 ? (i >= 3) : i / LE;
                const int w = LA == 2 ? 2 * u + v : u + v;
                acc[w] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[kk][u], b[kk][v], acc[w], 0, 0, 0);
                // fetch e follows MFMA (e * 4 LE) / FW of the step
                const int mi = kk * 2 * LE + i;
#pragma unroll
                for (int e = 0; e < FW; e++)
                    if (mi == (e * 4 * LE) / FW && more) issue1(qn, sn, e);
            }
        }
    }
}

// 64 x 64 output tile per block; wave (wr, wc) owns the 32 x 32 sub-tile,
// and each limb pair (u, v) accumulates apart, so the MFMAs of a step do not
// wait on each other.  Tiles are ordered so that the blocks on one XCD
// (block b runs on XCD b mod 8) share columns of B.  An int32 tile whose
// rows' top planes are all zero (rowlimb) runs the loop over three planes.
//
// Workgroups past the last tile run the last rounds of the product's
// sum-check instance (tail.hpp), which needs only the bound vectors, in the
// stage area's LDS: the single-workgroup tail then runs beside the tiles
// instead of after them.
template <int LA, int S, bool WIT>
__global__ __launch_bounds__(256, 2) void k_gemm_mfma(const int8_t *__restrict__ Al, const int8_t *__restrict__ Bt,
                                                   const int64_t *__restrict__ rowsum,
                                                   const int32_t *__restrict__ rowlimb,
                                                   const int64_t *__restrict__ colpart, int ntiles, uint32_t n,
                                                   uint32_t m, uint32_t k, uint32_t np, uint32_t mp, uint32_t kp,
                                                   int64_t *__restrict__ C, TailArgs ta, XJobs jobs, WitEpi we)
{
    static_assert(m61::block_sum_words(4, 256) * 8 <= S * (2 * (2 * LA + 4)) * 1024, "claims sum in the stage area");
    constexpr int F = 2 * (2 * LA + 4);
    static_assert(kTailSmem * 8 <= S * F * 1024, "the tail fits the stage area");
    __shared__ __attribute__((aligned(1024))) int8_t stage[S][F][1024];
    __shared__ int64_t s_cs[4][kTile], s_rs[kTile];
    __shared__ uint64_t s_e1[kTile];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wr = wv >> 1, wc = wv & 1, half = lane >> 5;
    const uint32_t nbi = np / kTile, nblk = nbi * (kp / kTile);
    if (blockIdx.x >= nblk) {  // workgroup-uniform
        tail_block<KIND_MATMUL>(ta, jobs, (int)(blockIdx.x - nblk), (uint64_t *)&stage[0][0][0]);
        return;
    }
    uint32_t t = blockIdx.x;
    if ((nblk & 7) == 0) t = (blockIdx.x & 7) * (nblk >> 3) + (blockIdx.x >> 3);
    const uint32_t bi = t % nbi, bj = t / nbi, i0 = bi * kTile, j0 = bj * kTile;
    const uint32_t nR = np >> 5, nC = kp >> 5, nQ = mp >> 5, nS = mp >> 6;
    // column sums of this block's columns over all row tiles of B (wave w takes
    // tiles w, w + 4, ...) and the row sums of its rows: loads issued first,
    // values used after the loop
    // (up to 64 row tiles: every load is issued before any is waited for,
    // one round trip in all; more tiles go through a loop)
    constexpr int kColRegs = 16;
    int64_t cs[4] = {0, 0, 0, 0}, rs = 0, cv[kColRegs];
    const bool col_regs = ntiles <= 4 * kColRegs;
#pragma unroll
    for (int e = 0; e < kColRegs; e++) cv[e] = 0;
    if (j0 + lane < k) {
        if (col_regs) {
#pragma unroll
            for (int e = 0; e < kColRegs; e++)
                if (wv + 4 * e < ntiles) cv[e] = colpart[(size_t)(wv + 4 * e) * kp + j0 + lane];
        } else {
            int ti = wv;
            for (; ti + 12 < ntiles; ti += 16)
#pragma unroll
                for (int q = 0; q < 4; q++) cs[q] += colpart[(size_t)(ti + 4 * q) * kp + j0 + lane];
            for (; ti < ntiles; ti += 4) cs[0] += colpart[(size_t)ti * kp + j0 + lane];
        }
    }
    if (tid < kTile && i0 + tid < n) rs = rowsum[i0 + tid];
    // the eq values of the witness claims (E1 of the tile's rows, E2 of this
    // lane's column), fetched before the loop so that the epilogue waits on
    // no load
    const int cl = 32 * wc + (lane & 31);
    const uint32_t col = j0 + cl;
    uint64_t e1own = 0, e2 = 0;
    if (WIT) {
        if (tid < kTile && i0 + tid < n) e1own = we.E1[i0 + tid];
        if (col < k) e2 = we.E2[col];
    }
    // limbs of each row (int32 A): does any row of the tile need plane 3
    int rl = 2;
    if (LA == 4) rl = tid < kTile && i0 + tid < n ? rowlimb[i0 + tid] : 3;
    // accumulators: int16 A, one per limb pair (index 2 u + v); int32 A, one per
    // weight u + v
    constexpr int NACC = LA == 2 ? 4 : LA + 1;
    v16i acc[NACC];
#pragma unroll
    for (int w = 0; w < NACC; w++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[w][r] = 0;
    if (LA == 4) {
        if (__syncthreads_or(rl > 3)) gemm_loop<LA, LA, S>(Al, Bt, bi, bj, nR, nC, nQ, nS, &stage[0][0][0], acc);
        else gemm_loop<LA, 3, S>(Al, Bt, bi, bj, nR, nC, nQ, nS, &stage[0][0][0], acc);
    } else {
        gemm_loop<LA, LA, S>(Al, Bt, bi, bj, nR, nC, nQ, nS, &stage[0][0][0], acc);
    }
#pragma unroll
    for (int e = 0; e < kColRegs; e++) cs[e & 3] += cv[e];
    s_cs[wv][lane] = cs[0] + cs[1] + cs[2] + cs[3];
    if (tid < kTile) {
        s_rs[tid] = rs;
        s_e1[tid] = e1own;
    }
    __syncthreads();
    // recombination in wrap-around 64-bit arithmetic: exact because C itself fits int64
    constexpr int64_t cA = LA == 2 ? 128 : 128 + 128 * 256 + 128 * 65536;
    const int64_t colsum = s_cs[0][cl] + s_cs[1][cl] + s_cs[2][cl] + s_cs[3][cl];
    const uint64_t corr = (uint64_t)cA * (uint64_t)colsum - (uint64_t)(128 * cA) * m;
    // With the witness fused (WIT) each entry also gives R, Rm, Y, Z and the
    // bit word, and the tile's claims at (r1, r2) and its range flag go to the
    // tile's partial (claims.hpp).  A lane's entries share its column, so the
    // lane sums E1[row] z over its sixteen rows and multiplies by E2[col]
    // once: E1 is cut into 21-bit limbs, so every limb sum is exact in int64
    // (|limb z| < 2^52).  Rows past n have E1 = 0 and columns past k E2 = 0,
    // so only the stores and the range flag need the bounds.  Z~ follows from
    // R~ and Y~: max(R, 0) = (R + |R|) / 2 under ReLU, Z = R otherwise.
    int64_t cl3[3][3] = {{0, 0, 0}, {0, 0, 0}, {0, 0, 0}};  // [claim R, Rm, Y][limb]
    int oor = 0;
    // Stores address the tile's first entry plus a 32-bit byte offset when
    // 64 rows of 8-byte entries span less than 2^32 bytes.
    const bool off32 = k < (1u << 23);
    const size_t tb = (size_t)i0 * k + j0;
    const uint32_t xo0 = (32 * wr + 4 * half) * k + cl;
#pragma unroll
    for (int r = 0; r < 16; r++) {
        const uint32_t lrow = 32 * wr + 8 * (r / 4) + 4 * half + (r % 4), row = i0 + lrow;
        const bool ok = row < n && col < k;
        uint64_t c = corr + 128 * (uint64_t)s_rs[lrow];
#pragma unroll
        for (int w = 0; w < NACC; w++) {
            const int wt = LA == 2 ? (w >> 1) + (w & 1) : w;  // weight 256^wt
            c += (uint64_t)(int64_t)acc[w][r] << (8 * wt);
        }
        WitOut o{};
        if (WIT) {
            int bad = 0;
            o = witness_entry((int64_t)c, we.s, we.t, we.relu, we.half, bad);
            oor |= ok ? bad : 0;
            const uint64_t e1 = s_e1[lrow];  // canonical, 0 past n
            const int32_t l0 = (int32_t)(e1 & 0x1FFFFF), l1 = (int32_t)((e1 >> 21) & 0x1FFFFF), l2 = (int32_t)(e1 >> 42);
            const int32_t z[3] = {o.r, o.rm, o.y};
#pragma unroll
            for (int q = 0; q < 3; q++) {
                cl3[q][0] += (int64_t)l0 * z[q];
                cl3[q][1] += (int64_t)l1 * z[q];
                cl3[q][2] += (int64_t)l2 * z[q];
            }
        }
        if (ok) {
            const uint32_t xo = xo0 + (8 * (r / 4) + (r % 4)) * k;  // entry offset within the tile
            if (off32) {
                *(int64_t *)((char *)(C + tb) + (xo << 3)) = (int64_t)c;
                if (WIT) {
                    *(int32_t *)((char *)(we.R + tb) + (xo << 2)) = o.r;
                    *(uint16_t *)((char *)(we.Rm + tb) + (xo << 1)) = (uint16_t)o.rm;
                    *(int32_t *)((char *)(we.Y + tb) + (xo << 2)) = o.y;
                    *(int32_t *)((char *)(we.Z + tb) + (xo << 2)) = o.z;
                    *(uint64_t *)((char *)(we.bits + tb) + (xo << 3)) = o.w;
                }
            } else {
                const size_t x = tb + xo;
                C[x] = (int64_t)c;
                if (WIT) {
                    we.R[x] = o.r;
                    we.Rm[x] = (uint16_t)o.rm;
                    we.Y[x] = o.y;
                    we.Z[x] = o.z;
                    we.bits[x] = o.w;
                }
            }
        }
    }
    if (WIT) {  // the stage area is free: every wave has passed the barrier above
        uint64_t cacc[3];
#pragma unroll
        for (int q = 0; q < 3; q++) {
            const uint64_t v = m61::fold(m61::from_i64(cl3[q][0]) + m61::rotl(m61::from_i64(cl3[q][1]), 21) +
                                         m61::rotl(m61::from_i64(cl3[q][2]), 42));
            cacc[q] = m61::lmul(v, e2);
        }
        const int any = __syncthreads_or(oor);
        m61::block_sum<3>(cacc, (uint64_t *)&stage[0][0][0]);
        if (tid == 0) {
            const uint64_t z = we.relu ? m61::rotl(m61::add(cacc[0], cacc[2]), 60) : cacc[0];  // 2^60 = 1/2
#pragma unroll
            for (int q = 0; q < 3; q++) we.claim_part[4 * (size_t)blockIdx.x + q] = cacc[q];
            we.claim_part[4 * (size_t)blockIdx.x + 3] = z;
            we.flags[blockIdx.x] = (uint32_t)any;
        }
    }
}

size_t gemm_workspace_bytes(int a_is_i32, uint32_t n, uint32_t m, uint32_t k)
{
    const size_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2;
    return LA * np * mp + 2 * kp * mp + 8 * (size_t)n + 4 * (size_t)np + 8 * (mp / 64) * kp + 4 * 256;
}

struct GemmWs {
    int8_t *Al, *Bt;
    int64_t *rowsum, *colpart;
    int32_t *rowlimb;
};

static GemmWs gemm_ws(void *ws, int LA, uint32_t n, uint32_t np, uint32_t mp, uint32_t kp)
{
    char *p = (char *)ws;
    GemmWs w;
    w.Al = (int8_t *)p;
    p += ((size_t)LA * np * mp + 255) & ~(size_t)255;
    w.Bt = (int8_t *)p;
    p += ((size_t)2 * kp * mp + 255) & ~(size_t)255;
    w.rowsum = (int64_t *)p;
    p += ((size_t)8 * n + 255) & ~(size_t)255;
    w.rowlimb = (int32_t *)p;
    p += ((size_t)4 * np + 255) & ~(size_t)255;
    w.colpart = (int64_t *)p;
    return w;
}

bool front_supported(int a_is_i32, uint32_t n, uint32_t m, uint32_t k, const void *A, const void *B)
{
    (void)a_is_i32;
    auto lg = [](uint32_t x) { int l = 0; while ((1u << l) < x) l++; return l; };
    return lg(n) <= kFrontMaxLog && lg(k) <= kFrontMaxLog && m >= 64 && k >= 8 && ((uintptr_t)A & 15) == 0 &&
           ((uintptr_t)B & 15) == 0;
}

void launch_front(const void *A, int a_is_i32, const int16_t *B, uint32_t n, uint32_t m, uint32_t k,
                  const uint64_t *r1, int ln, const uint64_t *r2, int lk, uint64_t *acc, uint64_t *b, uint64_t *E1,
                  uint64_t *E2, void *ws, hipStream_t st)
{
    const uint32_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2;
    const GemmWs w = gemm_ws(ws, LA, n, np, mp, kp);
    FrontArgs f{};
    f.A = A;
    f.B = B;
    f.n = n;
    f.m = m;
    f.k = k;
    f.np = np;
    f.mp = mp;
    f.kp = kp;
    f.Al = w.Al;
    f.rowsum = w.rowsum;
    f.rowlimb = w.rowlimb;
    f.Bt = w.Bt;
    f.colpart = w.colpart;
    f.r1 = r1;
    f.r2 = r2;
    f.ln = ln;
    f.lk = lk;
    f.acc = acc;
    f.b = b;
    f.E1 = E1;
    f.E2 = E2;
    // Row binding: about eight rows per lane and chunk (256 rows for int16,
    // 128 for int32), fewer (down to one per lane) while the role has under
    // 256 workgroups, so that a small matrix still spreads over the CUs.
    // Column binding: four rows per wave, one while that gives under 256
    // workgroups.
    constexpr uint32_t kFrontFill = 256;
    const uint32_t rs = a_is_i32 ? 16 : 32;  // row slots of a row-binding workgroup
    f.rpc = a_is_i32 ? 128 : 256;
    while (f.rpc > rs && (m / 64) * ((n + f.rpc - 1) / f.rpc) < kFrontFill) f.rpc >>= 1;
    f.n_rb = (m / 64) * ((n + f.rpc - 1) / f.rpc);
    const int rw = (m + 15) / 16 >= kFrontFill ? 4 : 1;
    f.n_cb = (m + 4 * rw - 1) / (4 * rw);
    f.n_sb = (kp / 64) * (mp / 64);
    f.n_sa = (np + 3) / 4;
    f.n_e1 = (n + 1023) / 1024;
    const uint32_t n_e2 = (k + 1023) / 1024;
    const dim3 grid(f.n_rb + f.n_cb + f.n_sb + f.n_sa + f.n_e1 + n_e2);
    if (a_is_i32) {
        if (rw == 4) hipLaunchKernelGGL((k_front<int32_t, 4, 4>), grid, dim3(256), 0, st, f);
        else hipLaunchKernelGGL((k_front<int32_t, 4, 1>), grid, dim3(256), 0, st, f);
    } else {
        if (rw == 4) hipLaunchKernelGGL((k_front<int16_t, 2, 4>), grid, dim3(256), 0, st, f);
        else hipLaunchKernelGGL((k_front<int16_t, 2, 1>), grid, dim3(256), 0, st, f);
    }
}

uint32_t gemm_tiles(uint32_t n, uint32_t k) { return (round_up64(k) / kTile) * (round_up64(n) / kTile); }

void launch_gemm_mfma(const void *A, int a_is_i32, const int16_t *B, int64_t *C, uint32_t n, uint32_t m, uint32_t k,
                      void *ws, hipStream_t st, const TailArgs *ta, const XJobs *jobs, bool split_done,
                      const WitEpi *we)
{
    const uint32_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2, ntiles = (int)(mp / 64);
    const GemmWs w = gemm_ws(ws, LA, n, np, mp, kp);
    const uint32_t na = (np + 3) / 4, nb = (kp / 64) * (mp / 64);
    if (!split_done) {
        if (a_is_i32)
            hipLaunchKernelGGL((k_split<int32_t, 4>), dim3(na + nb), dim3(256), 0, st, (const int32_t *)A, n, m, np,
                               mp, w.Al, w.rowsum, w.rowlimb, na, B, k, kp, w.Bt, w.colpart);
        else
            hipLaunchKernelGGL((k_split<int16_t, 2>), dim3(na + nb), dim3(256), 0, st, (const int16_t *)A, n, m, np,
                               mp, w.Al, w.rowsum, w.rowlimb, na, B, k, kp, w.Bt, w.colpart);
    }
    // tail workgroups (and the slot assemblies they bring) after the tiles
    const TailArgs tnone{};
    XJobs jnone{};
    const uint32_t extra = ta ? 1u + (uint32_t)jobs->nslot : 0u;
    const dim3 grid((kp / kTile) * (np / kTile) + extra);
    const TailArgs &tav = ta ? *ta : tnone;
    const XJobs &jv = ta ? *jobs : jnone;
    const WitEpi wnone{};
    const WitEpi &wv = we ? *we : wnone;
#define RA_GEMM(LAV, W)                                                                                            \
    hipLaunchKernelGGL((k_gemm_mfma<LAV, gemm_stages<LAV>(), W>), grid, dim3(256), 0, st, (const int8_t *)w.Al,    \
                       (const int8_t *)w.Bt, (const int64_t *)w.rowsum, (const int32_t *)w.rowlimb,                \
                       (const int64_t *)w.colpart, ntiles, n, m, k, np, mp, kp, C, tav, jv, wv)
    if (a_is_i32) {
        if (we) RA_GEMM(4, true);
        else RA_GEMM(4, false);
    } else {
        if (we) RA_GEMM(2, true);
        else RA_GEMM(2, false);
    }
#undef RA_GEMM
}

}  // namespace ra
