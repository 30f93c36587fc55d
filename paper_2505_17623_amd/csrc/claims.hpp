// claims.hpp -- the last step of the rescale / ReLU witness (Sec. II-A,
// III-B): the claims R~, Rm~, Y~, Z~ at (r1, r2) summed from the workgroups'
// partials, and (with the range parameter t given by the caller) the status
// from the workgroups' range flags.  Run by the witness's own one-workgroup
// launch, or by a workgroup of the range call's set-up launch when the
// witness call defers it.
#pragma once
#include "common.hpp"
#include "m61.hpp"
#include "ra.h"

namespace ra {

// Claims of V outputs: sum_i e_i z_i for e_i = E1[row] E2[col]
// (folded, < 2^61 + 8) and integers |z_i| <= 2^30 (R, Y, Z fit t <= 29; a
// value outside the given range makes the call fail, its claims unused).
// Each e_i is cut as e_hi 2^31 + e_lo, the two sums are exact in int64 (four
// terms below 2^61 each), then reduced mod p once.
template <int V>
__device__ __forceinline__ uint64_t claim_terms(const uint64_t (&el)[V], const uint64_t (&eh)[V],
                                                const int32_t (&z)[V])
{
    uint64_t lo = 0, hi = 0;  // two's complement sums (exact for |z| <= 2^30)
#pragma unroll
    for (int i = 0; i < V; i++) {
        lo += (uint64_t)((int64_t)el[i] * z[i]);
        hi += (uint64_t)((int64_t)eh[i] * z[i]);
    }
    return m61::fold(m61::from_i64((int64_t)lo) + m61::rotl(m61::from_i64((int64_t)hi), 31));
}

// One output of the rescale / ReLU witness (Sec. II-A, III-B) from its
// product entry c: R = floor((c + half) / 2^s), the shifted remainder Rm,
// Y = |R|, Z = ReLU(R) (or R), and the bit word (planes of Rm, R + 2^(t+1)
// and, with ReLU, Y).  *oor is set when R lies outside [-2^(t+1), 2^(t+1)).
struct WitOut {
    int32_t r, rm, y, z;
    uint64_t w;
};
__device__ __forceinline__ WitOut witness_entry(int64_t c, int s, int t, int relu, int64_t half, int &oor)
{
    WitOut o;
    const int64_t cc = c + half;
    const int64_t q = cc >> s;
    // qb = R + 2^(t+1): R lies in [-2^(t+1), 2^(t+1)) iff 0 <= qb < 2^(t+2)
    const int64_t qb = q + ((int64_t)1 << (t + 1));
    oor |= ((uint64_t)qb >> (t + 2)) != 0;
    o.rm = (int32_t)((uint32_t)cc & ((1u << s) - 1u));  // cc - 2^s floor(cc / 2^s), s <= 16
    o.r = (int32_t)q;
    o.y = o.r < 0 ? -o.r : o.r;
    o.z = relu ? (o.r > 0 ? o.r : 0) : o.r;
    o.w = (uint64_t)o.rm | ((uint64_t)qb << s);
    if (relu) o.w |= (uint64_t)o.y << (s + t + 2);
    return o;
}

// red: m61::block_sum_words(4, blockDim.x) words of LDS; res (LDS, optional):
// receives the parameters (words 0-7) and the claims (8-11), visible to the
// workgroup after the function's last barrier.
__device__ __forceinline__ void claims_final_block(const ClaimsJob &j, uint64_t *red, uint64_t *res)
{
    WitParams p;
    if (j.known) {  // the status from the workgroups' range flags; the parameters for the range call
        int any = 0;
        for (int b = threadIdx.x; b < j.nblk; b += blockDim.x) any |= j.flags[b] != 0;
        p = j.hp;
        if (__syncthreads_or(any)) p.status = RA_E_RANGE;
        if (threadIdx.x == 0) *j.prm = p;
    } else {
        p = *j.prm;
    }
    uint64_t acc[4] = {0, 0, 0, 0};
    if (p.status == 0)
        for (int b = threadIdx.x; b < j.nblk; b += blockDim.x)
            for (int i = 0; i < 4; i++) acc[i] = m61::add(acc[i], j.part[4 * b + i]);
    m61::block_sum<4>(acc, red);
    if (threadIdx.x == 0) {
        if (p.status == 0)
            for (int i = 0; i < 4; i++) j.out[i] = acc[i];
        uint64_t w[12];
        const uint64_t *pw = (const uint64_t *)&p;
        for (int i = 0; i < 8; i++) w[i] = i * 8 < (int)sizeof(WitParams) ? pw[i] : 0;
        for (int i = 0; i < 4; i++) w[8 + i] = acc[i];
        if (j.mirror)
            for (int i = 0; i < 12; i++) j.mirror[i] = w[i];
        if (res)
            for (int i = 0; i < 12; i++) res[i] = w[i];
    }
    __syncthreads();
}

}  // namespace ra
