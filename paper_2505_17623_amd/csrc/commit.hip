// commit.hip -- Pedersen vector commitments P = sum_i v_i G_i on secp256k1
// (Sec. II-C commits a vector a as g^a; Sec. IV names the curve), for the
// integer tables of a layer.
//
// The values are small integers (the witness tables hold 16- or 32-bit
// entries, the bit table 64-bit words), so the product is split by the bits
// of |v|:  P = sum_k 2^k (B_k^+ - B_k^-),  B_k^+- = the sum of G_i over the
// i with v_i >= 0 (< 0) and bit k of |v_i| set.  Each (k, sign) slot is a
// plain masked sum of generators: its threads stride over the points and add
// the ones whose bit is set (one mixed Jacobian-affine addition each), so the
// work does not depend on how the values are distributed; partial sums are
// then added in a tree, and one thread combines the slots by Horner's rule
// (a doubling per bit) and converts to affine coordinates.
#include <algorithm>

#include "commit.hpp"
#include "secp256k1.hpp"
#include "sha256.hpp"

namespace ra {

using secp::Aff;
using secp::Fe;
using secp::Jac;

// ---------------------------------------------------------------------------
// Generators by try-and-increment: x = SHA-256(tag || domain || LE64(i) ||
// LE32(c)) big-endian mod q for c = 0, 1, ...; the first x with x^3 + 7 a
// square gives (x, y), y the even root.
// ---------------------------------------------------------------------------
struct GenArgs {
    uint8_t domain[32];
    uint64_t first, count;
    uint32_t *gens, *err;
};

__global__ __launch_bounds__(256) void k_commit_generators(GenArgs a)
{
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.count) return;
    const uint64_t idx = a.first + i;
    const char tag[] = "range-arithmetic generators v1";
    for (uint32_t c = 0; c < 256; c++) {
        sha::Hasher h;
        h.init();
        h.update((const uint8_t *)tag, sizeof(tag) - 1);
        h.update(a.domain, 32);
        h.le(idx, 8);
        h.le(c, 4);
        uint8_t d[32];
        h.final(d);
        Fe x;
        for (int l = 0; l < 8; l++)
            x.v[l] = ((uint32_t)d[31 - 4 * l - 3] << 24) | ((uint32_t)d[31 - 4 * l - 2] << 16) |
                     ((uint32_t)d[31 - 4 * l - 1] << 8) | d[31 - 4 * l];
        x = secp::fe_canon(x, 0);
        const Fe rhs = secp::fe_add(secp::fe_mul(secp::fe_sqr(x), x), secp::fe_small(7));
        Fe y = secp::fe_sqrt(rhs);
        if (!secp::fe_eq(secp::fe_sqr(y), rhs)) continue;
        if (y.v[0] & 1) y = secp::fe_neg(y);
        uint32_t *o = a.gens + 16 * i;
        for (int l = 0; l < 8; l++) {
            o[l] = x.v[l];
            o[8 + l] = y.v[l];
        }
        return;
    }
    atomicOr(a.err, 1u);
}

void launch_commit_generators(const uint8_t *domain, uint64_t first, uint64_t count, uint32_t *gens, uint32_t *err,
                              hipStream_t st)
{
    GenArgs a{};
    for (int i = 0; i < 32; i++) a.domain[i] = domain[i];
    a.first = first;
    a.count = count;
    a.gens = gens;
    a.err = err;
    hipLaunchKernelGGL(k_commit_generators, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, a);
}

// ---------------------------------------------------------------------------
// The bit slots
// ---------------------------------------------------------------------------
int msm_bits(int kind) { return kind == 2 ? 32 : (kind == 3 ? 64 : 16); }
int msm_signs(int kind) { return (kind == 0 || kind == 2) ? 2 : 1; }
constexpr size_t kJacWords = 24;

size_t msm_workspace_bytes(int kind)
{
    const size_t slots = (size_t)msm_bits(kind) * msm_signs(kind);
    size_t b = slots * kMsmThreadsPerSlot * kJacWords * 4;                      // the threads' partial sums
    b += slots * ((kMsmThreadsPerSlot + kMsmGroup - 1) / kMsmGroup) * kJacWords * 4;  // one reduction level
    return b + 256;
}

// |v| and its sign for value i
__device__ __forceinline__ void scalar(const void *vals, int kind, uint64_t i, uint64_t &mag, int &neg)
{
    int64_t s;
    switch (kind) {
    case 0: s = ((const int16_t *)vals)[i]; break;
    case 1: mag = ((const uint16_t *)vals)[i]; neg = 0; return;
    case 2: s = ((const int32_t *)vals)[i]; break;
    default: mag = ((const uint64_t *)vals)[i]; neg = 0; return;
    }
    neg = s < 0;
    mag = (uint64_t)(s < 0 ? -s : s);
}

__device__ __forceinline__ void store_jac(uint32_t *p, const Jac &j)
{
    for (int l = 0; l < 8; l++) {
        p[l] = j.X.v[l];
        p[8 + l] = j.Y.v[l];
        p[16 + l] = j.Z.v[l];
    }
}
__device__ __forceinline__ Jac load_jac(const uint32_t *p)
{
    Jac j;
    for (int l = 0; l < 8; l++) {
        j.X.v[l] = p[l];
        j.Y.v[l] = p[8 + l];
        j.Z.v[l] = p[16 + l];
    }
    return j;
}

// slot s = blockIdx.y: bit k = s mod bits of the values of sign s / bits
__global__ __launch_bounds__(256) void k_msm_bits(const void *__restrict__ vals, int kind, uint64_t n,
                                                  const uint32_t *__restrict__ gens, int bits,
                                                  uint32_t *__restrict__ part)
{
    const int slot = blockIdx.y, k = slot % bits, want_neg = slot / bits;
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    Jac acc = secp::jac_inf();
    for (uint64_t i = t; i < n; i += kMsmThreadsPerSlot) {
        uint64_t mag;
        int neg;
        scalar(vals, kind, i, mag, neg);
        if (neg != want_neg || !((mag >> k) & 1)) continue;
        Aff g;
        const uint32_t *gp = gens + 16 * i;
        for (int l = 0; l < 8; l++) {
            g.x.v[l] = gp[l];
            g.y.v[l] = gp[8 + l];
        }
        acc = secp::jac_add_aff(acc, g);
    }
    store_jac(part + ((size_t)slot * kMsmThreadsPerSlot + t) * kJacWords, acc);
}

// out[slot][j] = sum of in[slot][j G .. j G + G - 1] (count entries per slot in, stride in_stride)
__global__ __launch_bounds__(256) void k_msm_reduce(const uint32_t *__restrict__ in, int count, int in_stride,
                                                    uint32_t *__restrict__ out, int out_stride)
{
    const int slot = blockIdx.y;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    const int groups = (count + kMsmGroup - 1) / kMsmGroup;
    if (j >= groups) return;
    Jac acc = secp::jac_inf();
    for (int q = j * kMsmGroup; q < std::min(count, (j + 1) * kMsmGroup); q++)
        acc = secp::jac_add(acc, load_jac(in + ((size_t)slot * in_stride + q) * kJacWords));
    store_jac(out + ((size_t)slot * out_stride + j) * kJacWords, acc);
}

// P = sum_k 2^k (B_k^+ - B_k^-) by Horner's rule, then affine bytes
__global__ void k_msm_final(const uint32_t *__restrict__ sums, int stride, int bits, int signs,
                            uint8_t *__restrict__ out)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    Jac acc = secp::jac_inf();
    for (int k = bits - 1; k >= 0; k--) {
        acc = secp::jac_dbl(acc);
        acc = secp::jac_add(acc, load_jac(sums + (size_t)k * stride * kJacWords));
        if (signs == 2) acc = secp::jac_add(acc, secp::jac_neg(load_jac(sums + (size_t)(bits + k) * stride * kJacWords)));
    }
    uint8_t b[64];
    secp::jac_encode(acc, b);
    for (int i = 0; i < 64; i++) out[i] = b[i];
}

void launch_commit(const void *vals, int kind, uint64_t n, const uint32_t *gens, void *ws, uint8_t *out,
                   hipStream_t st)
{
    const int bits = msm_bits(kind), slots = bits * msm_signs(kind);
    uint32_t *p0 = (uint32_t *)ws;
    uint32_t *p1 = p0 + (size_t)slots * kMsmThreadsPerSlot * kJacWords;
    hipLaunchKernelGGL(k_msm_bits, dim3(kMsmThreadsPerSlot / 256, slots), dim3(256), 0, st, vals, kind, n, gens, bits,
                       p0);
    // tree: 8192 -> 512 -> 32 -> 2 -> 1 partial sums per slot, alternating between the two areas
    int count = kMsmThreadsPerSlot, stride_in = kMsmThreadsPerSlot;
    uint32_t *in = p0, *outp = p1;
    while (count > 1) {
        const int groups = (count + kMsmGroup - 1) / kMsmGroup;
        hipLaunchKernelGGL(k_msm_reduce, dim3((groups + 255) / 256, slots), dim3(256), 0, st, in, count, stride_in,
                           outp, groups);
        std::swap(in, outp);
        stride_in = groups;
        count = groups;
    }
    hipLaunchKernelGGL(k_msm_final, dim3(1), dim3(64), 0, st, in, stride_in, bits, msm_signs(kind), out);
}

}  // namespace ra
