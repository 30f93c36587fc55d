// m61.hpp -- arithmetic in F_p, p = 2^61 - 1, for gfx950 wave64 kernels.
//
// Elements are uint64 in [0, p).  A product of two elements is formed from
// four 32x32->64 partial products (the high limbs are below 2^29), and the
// 122-bit result is folded with 2^61 = 1 (mod p): 2^64 = 8 and
// x 2^32 = (x >> 29) 2^61 + (x mod 2^29) 2^32 = (x >> 29) + (x mod 2^29) 2^32.
// Every helper returns a canonical value.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace m61 {

constexpr uint64_t P = 0x1FFFFFFFFFFFFFFFull;

__device__ __forceinline__ uint64_t reduce64(uint64_t x)
{
    // any x < 2^64 -> [0, p)
    x = (x & P) + (x >> 61);
    return x >= P ? x - P : x;
}

__device__ __forceinline__ uint64_t add(uint64_t a, uint64_t b)
{
    uint64_t s = a + b;
    return s >= P ? s - P : s;
}

__device__ __forceinline__ uint64_t sub(uint64_t a, uint64_t b) { return a >= b ? a - b : a + P - b; }

__device__ __forceinline__ uint64_t neg(uint64_t a) { return a ? P - a : 0; }

__device__ __forceinline__ uint64_t mul(uint64_t a, uint64_t b)
{
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t lo = (uint64_t)a0 * b0;                          // < 2^64
    const uint64_t mid = (uint64_t)a0 * b1 + (uint64_t)a1 * b0;     // < 2^62
    const uint64_t hi = (uint64_t)a1 * b1;                          // < 2^58
    const uint64_t s = (hi << 3) + (mid >> 29) + ((mid & 0x1FFFFFFFull) << 32) + (lo & P) + (lo >> 61);
    return reduce64(s);                                             // s < 2^63
}

__device__ __forceinline__ uint64_t sqr(uint64_t a) { return mul(a, a); }

// Field element of a signed integer with |z| < 2^63.
__device__ __forceinline__ uint64_t from_i64(int64_t z)
{
    if (z >= 0) return reduce64((uint64_t)z);
    return neg(reduce64((uint64_t)(-z)));
}

// Field element of a signed 32-bit integer.
__device__ __forceinline__ uint64_t from_i32(int32_t z)
{
    return z >= 0 ? (uint64_t)z : P - (uint64_t)(-(int64_t)z);
}

// a * 2^k for a canonical a and 0 <= k < 61: 2^61 = 1, so the residue rotates.
__device__ __forceinline__ uint64_t rotl(uint64_t a, int k)
{
    const uint64_t r = ((a << k) & P) | (a >> (61 - k));
    return r == P ? 0 : r;
}

// e * z for a field element e and a signed integer |z| < 2^31.
__device__ __forceinline__ uint64_t mul_small(uint64_t e, int32_t z)
{
    const uint32_t az = z < 0 ? (uint32_t)(-(int64_t)z) : (uint32_t)z;
    const uint64_t lo = (uint64_t)(uint32_t)e * az;                 // < 2^63
    const uint64_t hi = (uint64_t)(uint32_t)(e >> 32) * az;         // < 2^60, weight 2^32
    const uint64_t s = (hi >> 29) + ((hi & 0x1FFFFFFFull) << 32) + (lo & P) + (lo >> 61);
    const uint64_t r = reduce64(s);
    return z < 0 ? neg(r) : r;
}

// eq(z, b) for a single variable: z b + (1 - z)(1 - b) with b in {0, 1}.
__device__ __forceinline__ uint64_t eq1_bit(uint64_t z, uint32_t b) { return b ? z : sub(1, z); }

// eq(z, X) = (1 - X) + z (2X - 1) for a small integer X.
__device__ __forceinline__ uint64_t eq1_small(uint64_t z, int X)
{
    return add(from_i64(1 - X), mul_small(z, 2 * X - 1));
}

// ---------------------------------------------------------------------------
// Loose residues for hot loops.  A loose value is any uint64 x with
// x < 2^62 + 2^32 (its high word at most 2^30); it stands for x mod p.  The
// helpers below return "folded" values, x < 2^61 + 8, so a sum of two folded
// values is again loose.  canon() gives the canonical residue.
// ---------------------------------------------------------------------------

// Any x < 2^64 to a folded value (2^61 = 1): (x mod 2^61) + (x >> 61) < 2^61 + 8.
__host__ __device__ __forceinline__ uint64_t fold(uint64_t x) { return (x & P) + (x >> 61); }

// The value itself, hidden from the optimiser (it then keeps the operation
// that consumes it in the form written).  The host version is the identity.
__device__ __forceinline__ uint64_t opaque(uint64_t x)
{
    asm("" : "+v"(x));
    return x;
}
__host__ __forceinline__ uint64_t opaque(uint64_t x) { return x; }

// Product of two loose values, folded.  With a1, b1 <= 2^30:
//   a b = hi 2^64 + mid 2^32 + lo,  hi = a1 b1 <= 2^60, mid < 2^63, lo < 2^64;
//   2^64 = 8, mid 2^32 = (mid >> 29) + (mid mod 2^29) 2^32, lo = (lo >> 61) + (lo mod 2^61),
// and the five terms sum below 2^63 + 2^62 + 2^34 < 2^64.
__host__ __device__ __forceinline__ uint64_t lmul(uint64_t a, uint64_t b)
{
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t lo = (uint64_t)a0 * b0;
    const uint64_t mid = (uint64_t)a0 * b1 + (uint64_t)a1 * b0;
    uint64_t hi = (uint64_t)a1 * b1;
    const uint32_t lh = (uint32_t)(lo >> 32);
    // (mid mod 2^29) 2^32 + (lo >> 61): disjoint bits, one 64-bit word
    uint64_t t = (uint64_t)(lh >> 29) | ((uint64_t)((uint32_t)mid & 0x1FFFFFFFu) << 32);
    hi = opaque(hi);  // hi 8 stays one multiply and a shifted add
    t = opaque(t);    // t stays one word
    const uint64_t s = (hi << 3) + (mid >> 29) + ((uint64_t)(uint32_t)lo | ((uint64_t)(lh & 0x1FFFFFFFu) << 32)) + t;
    return fold(s);
}

// a - b for loose a, b, folded: a + 4p - b lies in (0, 2^64).
__host__ __device__ __forceinline__ uint64_t lsub(uint64_t a, uint64_t b) { return fold(a + (4 * P - b)); }

// a + b for a, b < 2^63, folded.
__host__ __device__ __forceinline__ uint64_t ladd(uint64_t a, uint64_t b) { return fold(a + b); }

// Canonical residue of any x < 2^64.
__host__ __device__ __forceinline__ uint64_t canon(uint64_t x)
{
    x = fold(x);  // < 2^61 + 8
    return x >= P ? x - P : x;
}

// Wave64 sum of one field element per lane (every lane gets the total).
__device__ __forceinline__ uint64_t wave_sum(uint64_t v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = add(v, __shfl_xor(v, off, 64));
    return v;
}

// Inclusive prefix product over the 64 lanes of a wave (lane i gets
// v_0 v_1 ... v_i); six shift-and-multiply steps.
__device__ __forceinline__ uint64_t wave_prefix_mul(uint64_t v)
{
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t u = __shfl_up(v, off, 64);
        if (lane >= off) v = mul(v, u);
    }
    return v;
}

// LDS words block_sum<NV> needs for a block of nt threads (nt a multiple of 64).
__host__ __device__ constexpr int block_sum_words(int NV, int nt) { return NV * nt + NV * 16 + NV; }

// Block sum of NV values per thread (canonical or folded residues).  On
// return (after a barrier) the NV canonical totals are at the returned LDS
// address for every thread.  `lds` must hold block_sum_words(NV, blockDim.x)
// words.  The values are transposed through LDS and summed in two stages (16
// interleaved segments per value, then the segments); sums of four terms are
// added without reduction before each fold, so no thread runs a long chain of
// dependent modular additions.
template <int NV>
__device__ __forceinline__ const uint64_t *block_sum_lds(const uint64_t (&v)[NV], uint64_t *lds)
{
    const int nt = blockDim.x, tid = threadIdx.x, seg = nt >> 4;
#pragma unroll
    for (int q = 0; q < NV; q++) lds[q * nt + tid] = v[q];
    __syncthreads();
    uint64_t *l2 = lds + NV * nt, *l3 = l2 + NV * 16;
    for (int task = tid; task < NV * 16; task += nt) {
        const uint64_t *src = lds + (task >> 4) * nt + (task & 15);  // entries g, g + 16, g + 32, ...
        uint64_t a0 = 0, a1 = 0;
        for (int e = 0; e < seg; e += 4) {
            a0 = fold(a0 + src[16 * e] + src[16 * e + 32]);
            a1 = fold(a1 + src[16 * e + 16] + src[16 * e + 48]);
        }
        l2[task] = fold(a0 + a1);
    }
    __syncthreads();
    if (tid < NV) {
        const uint64_t *g = l2 + tid * 16;
        const uint64_t a = fold(g[0] + g[1] + g[2] + g[3]), b = fold(g[4] + g[5] + g[6] + g[7]);
        const uint64_t c = fold(g[8] + g[9] + g[10] + g[11]), d = fold(g[12] + g[13] + g[14] + g[15]);
        l3[tid] = canon(fold(a + b) + fold(c + d));
    }
    __syncthreads();
    return l3;
}

// As block_sum_lds; thread 0 ends with the totals in v[].
template <int NV>
__device__ __forceinline__ void block_sum(uint64_t (&v)[NV], uint64_t *lds)
{
    const uint64_t *t = block_sum_lds<NV>(v, lds);
    if (threadIdx.x == 0)
#pragma unroll
        for (int q = 0; q < NV; q++) v[q] = t[q];
    __syncthreads();
}

}  // namespace m61
