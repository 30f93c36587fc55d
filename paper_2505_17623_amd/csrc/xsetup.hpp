// xsetup.hpp -- set-up of the rounds over x (xrounds.hip): suffix eq tables
// and the prefix products K_j of the range and ReLU instances.
//   HS heap: table s (2^s entries at offset 2^s) = eq(r_{lN-L-s .. lN-L-1}, .)
//   LS heap: table s (2^s entries at offset 2^s) = eq(r_{lN-s .. lN-1}, .)
//   Kr[j] = prod_{l<j} eq1(r_l, sigma_x,l),  Kz[j] = prod_{l<j} eq1(r_l, rho'_l)
#pragma once
#include "common.hpp"
#include "m61.hpp"

namespace ra {

__device__ __forceinline__ uint64_t eq_suffix(const uint64_t *r, int first, int s, uint64_t i)
{
    uint64_t a = 1;
    for (int t = 0; t < s; t++) a = m61::mul(a, m61::eq1_bit(r[first + t], (uint32_t)(i >> (s - 1 - t)) & 1u));
    return a;
}

// Thread gid (0 .. x_setup_threads - 1) of the set-up.
__device__ __forceinline__ void x_setup_body(const XSetupArgs &a, int gid)
{
    const int lN = a.lN, L = a.L, nhs = a.nhs, nls = 1 << (L + 1);
    if (gid < 128) {  // waves 0 and 1: prefix products of the two instances (lN < 64)
        const uint64_t *z = gid < 64 ? a.sigx : a.rho2;
        uint64_t *K = gid < 64 ? a.Kr : a.Kz;
        const int j = gid & 63;
        if (z) {  // wave-uniform
            uint64_t e = 1;
            if (j < lN) e = m61::add(m61::mul(a.r[j], z[j]), m61::mul(m61::sub(1, a.r[j]), m61::sub(1, z[j])));
            const uint64_t inc = m61::wave_prefix_mul(e);  // prod_{l <= j}
            if (j < lN) K[j + 1] = inc;
            if (j == 0) K[0] = 1;
        }
    }
    if (gid == 1) a.HS[0] = a.LS[0] = 0;  // unused heap slots
    if (gid >= 1 && gid < nhs) {
        const int s = 31 - __clz(gid);
        a.HS[gid] = eq_suffix(a.r, lN - L - s, s, (uint64_t)(gid - (1 << s)));
    }
    const int e = gid - nhs;
    if (e >= 1 && e < nls) {
        const int s = 31 - __clz(e);
        a.LS[e] = eq_suffix(a.r, lN - s, s, (uint64_t)(e - (1 << s)));
    }
}

}  // namespace ra
