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
