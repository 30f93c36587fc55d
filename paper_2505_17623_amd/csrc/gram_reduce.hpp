// gram_reduce.hpp -- the sum of the Gram pass's per-block partial tiles
// (plane rounds of the concatenated range check, Sec. III-B), shared by the
// reduction launch and the extra workgroups of the first x-round launch that
// run it beside the rounds.
#pragma once
#include "common.hpp"
#include "m61.hpp"

namespace ra {

// Output fragment of v_mfma_i32_16x16x64_i8: lane l, register r holds
// row 4 (l / 16) + r, column l % 16 of the 16 x 16 tile.
__host__ __device__ constexpr int frag_row(int l, int r) { return 4 * (l / 16) + r; }

// The 16 x 16 tiles on and above the diagonal of the symmetric Gram matrix,
// over nb blocks of sixteen planes (nb (nb + 1) / 2 tiles): tile t covers
// blocks (I, J), I <= J, in the order (0,0), (0,1), .., (0,nb-1), (1,1), ..
__device__ __forceinline__ void tile_blocks(int t, int nb, int &I, int &J)
{
    I = 0;
    while (t >= nb - I) {
        t -= nb - I;
        I++;
    }
    J = I + t;
}

// Workgroup blk (256 threads) of the reduction: 16 entries of G, sixteen
// lanes per entry (lane group g sums the partial tiles of blocks g, g + 16,
// ...), then LDS; G[q][q'] is written in both triangles.  With 6 tiles (48
// of 64 planes) the workgroups also clear the rest of the 64 x 64 matrix
// (96 workgroups, 240 spare threads each, for 1792 entries).
constexpr int kGramReduceLdsWords = 16 * 17;
__device__ __forceinline__ void gram_reduce_block(const uint64_t *__restrict__ gpart, int nblk, int tiles,
                                                  uint64_t *__restrict__ G, int blk, uint64_t *lds)
{
    uint64_t(*red)[17] = (uint64_t(*)[17])lds;
    const int tid = threadIdx.x, el = tid & 15, g = tid >> 4, entries = tiles * kGramTileWords;
    const int e = blk * 16 + el;
    uint64_t a = 0;
    int b = g;
    for (; b + 48 < nblk; b += 64) {  // four partials per iteration, loads first, one fold
        const uint64_t v0 = gpart[(size_t)b * entries + e], v1 = gpart[(size_t)(b + 16) * entries + e];
        const uint64_t v2 = gpart[(size_t)(b + 32) * entries + e], v3 = gpart[(size_t)(b + 48) * entries + e];
        a = m61::fold(a + v0 + v1 + v2 + v3);
    }
    for (; b < nblk; b += 16) a = m61::fold(a + gpart[(size_t)b * entries + e]);
    red[g][el] = a;
    if (tiles == 6 && tid >= 16) {  // 48 planes: G's rows and columns of planes 48 .. 63 are zero
        const int z = blk * 240 + (tid - 16);  // 16 x 64 entries of the rows, then 48 x 16 of the columns
        if (z < 16 * 64 + 48 * 16) {
            const int q = z < 1024 ? 48 + (z >> 6) : (z - 1024) >> 4;
            const int q2 = z < 1024 ? (z & 63) : 48 + ((z - 1024) & 15);
            G[q * 64 + q2] = 0;
        }
    }
    __syncthreads();
    if (tid >= 16) return;
    uint64_t v = 0;
#pragma unroll
    for (int q = 0; q < 16; q += 4) v = m61::fold(v + red[q][el] + red[q + 1][el] + red[q + 2][el] + red[q + 3][el]);
    v = m61::canon(v);
    const int t = e / kGramTileWords, r = (e % kGramTileWords) >> 6, l = e & 63;
    int I, J;
    tile_blocks(t, tiles == 3 ? 2 : (tiles == 6 ? 3 : 4), I, J);  // 3 tiles: 32 planes; 6: 48; 10: 64
    const int q = 16 * I + frag_row(l, r), q2 = 16 * J + (l & 15);
    G[q * 64 + q2] = v;
    G[q2 * 64 + q] = v;  // symmetric (the same value when the tile is diagonal)
}

}  // namespace ra
