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

namespace ra {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kTile = 64;   // block tile (rows and columns) and k-chunk
constexpr int kRowPad = 80; // LDS row stride in bytes (64 + 16)

__host__ __device__ inline uint32_t round_up64(uint32_t v) { return (v + 63u) & ~63u; }

// Byte gathers: v_perm_b32 picks bytes of {hi, lo} (selector bytes 0-3 from
// lo, 4-7 from hi, 0x0c gives zero).
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel)
{
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// A (n x m) -> limb planes Al[u][np][mp] (zero padded) and rowsum(A).  One
// wave per row; a lane takes 16 consecutive entries and writes 16 bytes per
// limb: the low byte shifted by -128 (a xor of the sign bit), the top limb
// as is.
template <typename TA, int LA>
__device__ __forceinline__ void split_a_block(const TA *__restrict__ A, uint32_t n, uint32_t m, uint32_t np,
                                              uint32_t mp, int8_t *__restrict__ Al, int64_t *__restrict__ rowsum,
                                              uint32_t blk)
{
    const uint32_t row = blk * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= np) return;  // wave-uniform
    const size_t plane = (size_t)np * mp;
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
#pragma unroll
        for (int u = 0; u < LA; u++) *(v4i *)&Al[u * plane + (size_t)row * mp + c] = out[u];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0 && row < n) rowsum[row] = s;
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
    const size_t plane = (size_t)kp * mp;
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
    *(v4i *)&Bt[(size_t)j * mp + l0 + ch] = o0;
    *(v4i *)&Bt[plane + (size_t)j * mp + l0 + ch] = o1;
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
                                               uint32_t na, const int16_t *__restrict__ B, uint32_t k, uint32_t kp,
                                               int8_t *__restrict__ Bt, int64_t *__restrict__ colpart)
{
    if (blockIdx.x < na) {
        split_a_block<TA, LA>(A, n, m, np, mp, Al, rowsum, blockIdx.x);
        return;
    }
    const uint32_t t = blockIdx.x - na, tx = kp / 64;
    split_bt_block(B, m, k, mp, kp, Bt, colpart, t % tx, t / tx);
}

// 64 x 64 output tile per block; wave (wr, wc) owns the 32 x 32 sub-tile.
template <int LA>
__global__ __launch_bounds__(256) void k_gemm_mfma(const int8_t *__restrict__ Al, const int8_t *__restrict__ Bt,
                                                   const int64_t *__restrict__ rowsum,
                                                   const int64_t *__restrict__ colpart, int ntiles, int64_t cA,
                                                   uint32_t n, uint32_t m, uint32_t k, uint32_t np, uint32_t mp,
                                                   uint32_t kp, int64_t *__restrict__ C)
{
    constexpr int W = LA + 1;  // limb weights 0 .. LA
    __shared__ __attribute__((aligned(16))) int8_t As[LA][kTile][kRowPad];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][kTile][kRowPad];
    __shared__ int64_t s_cs[4][kTile];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wr = wv >> 1, wc = wv & 1, half = lane >> 5;
    const uint32_t i0 = blockIdx.y * kTile, j0 = blockIdx.x * kTile;
    const size_t aplane = (size_t)np * mp, bplane = (size_t)kp * mp;
    {   // column sums of this block's columns over all row tiles of B: wave w takes tiles w, w + 4, ...
        int64_t cs[4] = {0, 0, 0, 0};
        if (j0 + lane < k) {
            int ti = wv;
            for (; ti + 12 < ntiles; ti += 16)
#pragma unroll
                for (int q = 0; q < 4; q++) cs[q] += colpart[(size_t)(ti + 4 * q) * kp + j0 + lane];
            for (; ti < ntiles; ti += 4) cs[0] += colpart[(size_t)ti * kp + j0 + lane];
        }
        s_cs[wv][lane] = cs[0] + cs[1] + cs[2] + cs[3];
    }
    v16i acc[W];
#pragma unroll
    for (int w = 0; w < W; w++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[w][r] = 0;
    const int lr = tid >> 2, lp = (tid & 3) * 16;  // staging: row, 16-byte piece
    for (uint32_t k0 = 0; k0 < mp; k0 += kTile) {
#pragma unroll
        for (int u = 0; u < LA; u++)
            *(v4i *)&As[u][lr][lp] = *(const v4i *)&Al[u * aplane + (size_t)(i0 + lr) * mp + k0 + lp];
#pragma unroll
        for (int v = 0; v < 2; v++)
            *(v4i *)&Bs[v][lr][lp] = *(const v4i *)&Bt[v * bplane + (size_t)(j0 + lr) * mp + k0 + lp];
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < 2; ks++) {
            const int ko = 32 * ks + 16 * half;
            v4i a[LA], b[2];
#pragma unroll
            for (int u = 0; u < LA; u++) a[u] = *(const v4i *)&As[u][32 * wr + (lane & 31)][ko];
#pragma unroll
            for (int v = 0; v < 2; v++) b[v] = *(const v4i *)&Bs[v][32 * wc + (lane & 31)][ko];
#pragma unroll
            for (int u = 0; u < LA; u++)
#pragma unroll
                for (int v = 0; v < 2; v++) acc[u + v] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[u], b[v], acc[u + v], 0, 0, 0);
        }
        __syncthreads();
    }
    // recombination in wrap-around 64-bit arithmetic: exact because C itself fits int64
    const int cl = 32 * wc + (lane & 31);
    const uint32_t col = j0 + cl;
    const int64_t colsum = s_cs[0][cl] + s_cs[1][cl] + s_cs[2][cl] + s_cs[3][cl];
    const uint64_t corr = (uint64_t)cA * (uint64_t)colsum - (uint64_t)(128 * cA) * m;
#pragma unroll
    for (int r = 0; r < 16; r++) {
        const uint32_t row = i0 + 32 * wr + 8 * (r / 4) + 4 * half + (r % 4);
        if (row < n && col < k) {
            uint64_t c = corr + 128 * (uint64_t)rowsum[row];
#pragma unroll
            for (int w = 0; w < W; w++) c += (uint64_t)(int64_t)acc[w][r] << (8 * w);
            C[(size_t)row * k + col] = (int64_t)c;
        }
    }
}

size_t gemm_workspace_bytes(int a_is_i32, uint32_t n, uint32_t m, uint32_t k)
{
    const size_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2;
    return LA * np * mp + 2 * kp * mp + 8 * (size_t)n + 8 * (mp / 64) * kp + 3 * 256;
}

void launch_gemm_mfma(const void *A, int a_is_i32, const int16_t *B, int64_t *C, uint32_t n, uint32_t m, uint32_t k,
                      void *ws, hipStream_t st)
{
    const uint32_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2, ntiles = (int)(mp / 64);
    char *p = (char *)ws;
    int8_t *Al = (int8_t *)p;
    p += ((size_t)LA * np * mp + 255) & ~(size_t)255;
    int8_t *Bt = (int8_t *)p;
    p += ((size_t)2 * kp * mp + 255) & ~(size_t)255;
    int64_t *rowsum = (int64_t *)p;
    p += ((size_t)8 * n + 255) & ~(size_t)255;
    int64_t *colpart = (int64_t *)p;
    const uint32_t na = (np + 3) / 4, nb = (kp / 64) * (mp / 64);
    if (a_is_i32)
        hipLaunchKernelGGL((k_split<int32_t, 4>), dim3(na + nb), dim3(256), 0, st, (const int32_t *)A, n, m, np, mp, Al,
                           rowsum, na, B, k, kp, Bt, colpart);
    else
        hipLaunchKernelGGL((k_split<int16_t, 2>), dim3(na + nb), dim3(256), 0, st, (const int16_t *)A, n, m, np, mp, Al,
                           rowsum, na, B, k, kp, Bt, colpart);
    const dim3 grid(kp / kTile, np / kTile);
    if (a_is_i32)
        hipLaunchKernelGGL(k_gemm_mfma<4>, grid, dim3(256), 0, st, (const int8_t *)Al, (const int8_t *)Bt,
                           (const int64_t *)rowsum, (const int64_t *)colpart, ntiles, (int64_t)8421504, n, m, k, np,
                           mp, kp, C);
    else
        hipLaunchKernelGGL(k_gemm_mfma<2>, grid, dim3(256), 0, st, (const int8_t *)Al, (const int8_t *)Bt,
                           (const int64_t *)rowsum, (const int64_t *)colpart, ntiles, (int64_t)128, n, m, k, np, mp,
                           kp, C);
}

}  // namespace ra
