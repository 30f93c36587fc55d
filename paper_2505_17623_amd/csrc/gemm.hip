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

// A (n x m) -> limb planes Al[u][np][mp] (zero padded) and rowsum(A); one wave per row.
template <typename TA, int LA>
__global__ __launch_bounds__(256) void k_split_a(const TA *__restrict__ A, uint32_t n, uint32_t m, uint32_t np,
                                                 uint32_t mp, int8_t *__restrict__ Al, int64_t *__restrict__ rowsum)
{
    const uint32_t row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= np) return;  // wave-uniform
    const size_t plane = (size_t)np * mp;
    int64_t s = 0;
    for (uint32_t c = lane * 4; c < mp; c += 256) {
        int8_t lb[LA][4];
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const bool in = row < n && c + e < m;
            const int32_t a = in ? (int32_t)A[(size_t)row * m + c + e] : 0;
            s += a;
#pragma unroll
            for (int u = 0; u < LA; u++) {
                int32_t d = u == LA - 1 ? (a >> (8 * u)) : (((a >> (8 * u)) & 255) - 128);
                lb[u][e] = in ? (int8_t)d : 0;
            }
        }
#pragma unroll
        for (int u = 0; u < LA; u++) {
            const uint32_t word = (uint32_t)(uint8_t)lb[u][0] | ((uint32_t)(uint8_t)lb[u][1] << 8) |
                                  ((uint32_t)(uint8_t)lb[u][2] << 16) | ((uint32_t)(uint8_t)lb[u][3] << 24);
            *(uint32_t *)&Al[u * plane + (size_t)row * mp + c] = word;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0 && row < n) rowsum[row] = s;
}

__global__ void k_zero_i64(int64_t *__restrict__ p, uint32_t len)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < len) p[i] = 0;
}

// B (m x k) -> transposed limb planes Bt[v][kp][mp] (row j holds column j of
// B, zero padded) and colsum(B); 64 x 64 tiles transposed through LDS.
__global__ __launch_bounds__(256) void k_split_bt(const int16_t *__restrict__ B, uint32_t m, uint32_t k, uint32_t mp,
                                                  uint32_t kp, int8_t *__restrict__ Bt,
                                                  unsigned long long *__restrict__ colsum)
{
    __shared__ int16_t t[64][65];
    const uint32_t l0 = blockIdx.y * 64, j0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const uint32_t l = l0 + r, j = j0 + tx;
        t[r][tx] = (l < m && j < k) ? B[(size_t)l * k + j] : (int16_t)0;
    }
    __syncthreads();
    const size_t plane = (size_t)kp * mp;
    // thread (tx = l offset, ty): columns j0 + ty + 4 i; write Bt[v][j][l0 + tx]
    for (int i = 0; i < 16; i++) {
        const int jj = ty + 4 * i;
        const uint32_t j = j0 + jj, l = l0 + tx;
        const int32_t b = t[tx][jj];
        const bool in = l < m && j < k;
        const int8_t b0 = in ? (int8_t)((b & 255) - 128) : 0, b1 = in ? (int8_t)(b >> 8) : 0;
        Bt[(size_t)j * mp + l] = b0;
        Bt[plane + (size_t)j * mp + l] = b1;
    }
    // column sums of this tile
    if (threadIdx.x < 64) {
        int64_t s = 0;
        for (int r = 0; r < 64; r++) s += t[r][threadIdx.x];
        if (j0 + threadIdx.x < k) atomicAdd(&colsum[j0 + threadIdx.x], (unsigned long long)s);
    }
}

// 64 x 64 output tile per block; wave (wr, wc) owns the 32 x 32 sub-tile.
template <int LA>
__global__ __launch_bounds__(256) void k_gemm_mfma(const int8_t *__restrict__ Al, const int8_t *__restrict__ Bt,
                                                   const int64_t *__restrict__ rowsum,
                                                   const unsigned long long *__restrict__ colsum, int64_t cA,
                                                   uint32_t n, uint32_t m, uint32_t k, uint32_t np, uint32_t mp,
                                                   uint32_t kp, int64_t *__restrict__ C)
{
    constexpr int W = LA + 1;  // limb weights 0 .. LA
    __shared__ __attribute__((aligned(16))) int8_t As[LA][kTile][kRowPad];
    __shared__ __attribute__((aligned(16))) int8_t Bs[2][kTile][kRowPad];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wr = wv >> 1, wc = wv & 1, half = lane >> 5;
    const uint32_t i0 = blockIdx.y * kTile, j0 = blockIdx.x * kTile;
    const size_t aplane = (size_t)np * mp, bplane = (size_t)kp * mp;
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
    const uint32_t col = j0 + 32 * wc + (lane & 31);
    const uint64_t corr = (col < k ? (uint64_t)cA * colsum[col] : 0) - (uint64_t)(128 * cA) * m;
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
    return LA * np * mp + 2 * kp * mp + 8 * (size_t)n + 8 * (size_t)k + 3 * 256;
}

void launch_gemm_mfma(const void *A, int a_is_i32, const int16_t *B, int64_t *C, uint32_t n, uint32_t m, uint32_t k,
                      void *ws, hipStream_t st)
{
    const uint32_t np = round_up64(n), mp = round_up64(m), kp = round_up64(k);
    const int LA = a_is_i32 ? 4 : 2;
    char *p = (char *)ws;
    int8_t *Al = (int8_t *)p;
    p += ((size_t)LA * np * mp + 255) & ~(size_t)255;
    int8_t *Bt = (int8_t *)p;
    p += ((size_t)2 * kp * mp + 255) & ~(size_t)255;
    int64_t *rowsum = (int64_t *)p;
    p += ((size_t)8 * n + 255) & ~(size_t)255;
    unsigned long long *colsum = (unsigned long long *)p;
    hipLaunchKernelGGL(k_zero_i64, dim3((k + 255) / 256), dim3(256), 0, st, (int64_t *)colsum, k);
    if (a_is_i32)
        hipLaunchKernelGGL((k_split_a<int32_t, 4>), dim3((np + 3) / 4), dim3(256), 0, st, (const int32_t *)A, n, m, np, mp, Al, rowsum);
    else
        hipLaunchKernelGGL((k_split_a<int16_t, 2>), dim3((np + 3) / 4), dim3(256), 0, st, (const int16_t *)A, n, m, np, mp, Al, rowsum);
    hipLaunchKernelGGL(k_split_bt, dim3(kp / 64, mp / 64), dim3(256), 0, st, B, m, k, mp, kp, Bt, colsum);
    const dim3 grid(kp / kTile, np / kTile);
    if (a_is_i32)
        hipLaunchKernelGGL(k_gemm_mfma<4>, grid, dim3(256), 0, st, (const int8_t *)Al, (const int8_t *)Bt,
                           (const int64_t *)rowsum, (const unsigned long long *)colsum, (int64_t)8421504, n, m, k, np,
                           mp, kp, C);
    else
        hipLaunchKernelGGL(k_gemm_mfma<2>, grid, dim3(256), 0, st, (const int8_t *)Al, (const int8_t *)Bt,
                           (const int64_t *)rowsum, (const unsigned long long *)colsum, (int64_t)128, n, m, k, np, mp,
                           kp, C);
}

}  // namespace ra
