// xsetup.hpp -- set-up of the rounds over x (xrounds.hip): suffix eq tables
// and the prefix products K_j of the range and ReLU instances.
//   HS heap: table s (2^s entries at offset 2^s) = eq(r_{lN-L-s .. lN-L-1}, .)
//   LS heap: table s (2^s entries at offset 2^s) = eq(r_{lN-s .. lN-1}, .)
//   WS heap: table s (2^s entries at offset 2^s, s < wB) = eq(r_{wj+wB-s .. wj+wB-1}, .),
//            the weights inside the sub-cubes of the LDS pass over rounds wj .. wj+wB-1
//   Kr[j] = prod_{l<j} eq1(r_l, sigma_x,l),  Kz[j] = prod_{l<j} eq1(r_l, rho'_l)
#pragma once
#include "common.hpp"
#include "m61.hpp"

namespace ra {

// eq(r[first .. first + s), i) with i's most significant of s bits first; r in LDS.
__device__ __forceinline__ uint64_t eq_suffix(const uint64_t *r, int first, int s, uint64_t i)
{
    uint64_t a = 1;
    for (int t = 0; t < s; t++) {
        const uint64_t z = r[first + t];
        a = m61::lmul(a, ((i >> (s - 1 - t)) & 1) ? z : m61::lsub(1, z));
    }
    return m61::canon(a);
}

// Threads of the set-up of an instance with lN variables.
__host__ __device__ inline int x_setup_count(const XSetupArgs &a)
{
    return (a.lN > a.L ? 1 << (a.lN - a.L) : 1) + (1 << (a.L + 1)) + (a.wB > 0 ? 1 << a.wB : 0);
}

// Thread gid (0 .. x_setup_count - 1) of the set-up; rl, zl: r and the two
// instances' challenges (sigma_x, rho'; lN words each) staged in LDS.
__device__ __forceinline__ void x_setup_body(const XSetupArgs &a, int gid, const uint64_t *rl, const uint64_t *sl,
                                             const uint64_t *zl)
{
    const int lN = a.lN, L = a.L, nhs = a.nhs, nls = 1 << (L + 1);
    if (gid < 128) {  // waves 0 and 1: prefix products of the two instances (lN < 64)
        const uint64_t *z = gid < 64 ? sl : zl;
        uint64_t *K = gid < 64 ? a.Kr : a.Kz;
        const int j = gid & 63;
        if (gid < 64 || a.rho2) {  // wave-uniform
            uint64_t e = 1;
            if (j < lN) e = m61::add(m61::mul(rl[j], z[j]), m61::mul(m61::sub(1, rl[j]), m61::sub(1, z[j])));
            const uint64_t inc = m61::wave_prefix_mul(e);  // prod_{l <= j}
            if (j < lN) K[j + 1] = inc;
            if (j == 0) K[0] = 1;
        }
    }
    if (gid == 1) a.HS[0] = a.LS[0] = 0;  // unused heap slots
    if (gid >= 1 && gid < nhs) {
        const int s = 31 - __clz(gid);
        a.HS[gid] = eq_suffix(rl, lN - L - s, s, (uint64_t)(gid - (1 << s)));
    }
    const int e = gid - nhs;
    if (e >= 1 && e < nls) {
        const int s = 31 - __clz(e);
        a.LS[e] = eq_suffix(rl, lN - s, s, (uint64_t)(e - (1 << s)));
    }
    const int w = e - nls;
    if (a.wB > 0 && w >= 0 && w < (1 << a.wB)) {
        if (w == 0) {
            a.WS[0] = 0;
        } else {
            const int s = 31 - __clz(w);
            a.WS[w] = eq_suffix(rl, a.wj + a.wB - s, s, (uint64_t)(w - (1 << s)));
        }
    }
}

}  // namespace ra
