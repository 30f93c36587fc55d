// commit.hip -- Pedersen vector commitments P = sum_i v_i G_i on secp256k1
// (Sec. II-C commits a vector a as g^a; Sec. IV names the curve), for the
// integer tables of a layer.
//
// The multi-scalar product is the bucket (Pippenger) method with 8-bit
// windows of |v_i| (two windows for 16-bit values, four for 32-bit, eight
// for 64-bit words), the sign applied to the point:
//   P = sum_w 2^(8w) sum_{b=1}^{255} b S_{w,b},  S_{w,b} = sum of sign(v_i) G_i
//   over the i whose window-w digit of |v_i| is b.
// A workgroup takes a chunk of values and one window: it sorts the chunk by
// digit in LDS (a counting sort), then every thread adds an equal run of the
// sorted list with mixed Jacobian-affine additions, so a heavy bucket is
// spread over many threads; the runs' partial sums, in bucket order, are
// added per bucket.  The chunks' bucket sums are then added per bucket, and
// sum_b b S_{w,b} is formed as sum_k 2^k (sum over the b with bit k set).
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
// The bucket method
// ---------------------------------------------------------------------------
constexpr int kPipSub = 4096;              // values a workgroup sorts at a time (two workgroups fit a CU)
constexpr int kPipParts = 256 + 255;       // run partials of one sort, at most
constexpr int kJacWords = 24;              // X, Y, Z: eight 32-bit limbs each

int msm_windows(int kind) { return kind == 3 ? 8 : (kind == 2 ? 4 : 2); }

size_t msm_workspace_bytes(int kind)
{
    const size_t W = (size_t)msm_windows(kind), jac = (size_t)kJacWords * 4;
    return W * kMsmChunks * 256 * jac   // the chunks' bucket sums
           + W * 256 * jac             // the bucket sums
           + W * 8 * jac               // their bit sums
           + 256;
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

// Exclusive prefix sums of one value per thread (256 threads); the total to
// *total.  sc: 4 words of LDS.
__device__ __forceinline__ uint32_t block_scan256(uint32_t v, uint32_t *sc, uint32_t *total)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t inc = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) sc[wv] = inc;
    __syncthreads();
    uint32_t before = 0;
    for (int q = 0; q < wv; q++) before += sc[q];
    if (total && threadIdx.x == 255) *total = before + inc;
    const uint32_t ex = before + inc - v;
    __syncthreads();
    return ex;
}

// Workgroup (c, w): the window-w bucket sums of values c L .. c L + L - 1
// (L = per), in sorts of kPipSub values; written to out[(w C + c) 256 + b].
__global__ __launch_bounds__(256) void k_pip_buckets(const void *__restrict__ vals, int kind, uint64_t n,
                                                     const uint32_t *__restrict__ gens, uint64_t per,
                                                     uint32_t *__restrict__ out)
{
    __shared__ uint8_t dig[kPipSub], sgn[kPipSub];
    __shared__ uint16_t perm[kPipSub];
    __shared__ uint32_t cnt[256], cur[256], first[256], sc[4], tot[2];
    __shared__ uint8_t pd[kPipParts];
    __shared__ uint32_t pp[kPipParts][kJacWords];
    const int tid = threadIdx.x, w = blockIdx.y, c = blockIdx.x;
    const uint64_t lo = (uint64_t)c * per, hi = lo + per < n ? lo + per : n;
    Jac bucket = secp::jac_inf();  // thread b's bucket b (b >= 1)
    for (uint64_t base = lo; base < hi; base += kPipSub) {
        const int len = (int)(hi - base < (uint64_t)kPipSub ? hi - base : (uint64_t)kPipSub);
        cnt[tid] = 0;
        first[tid] = 0xFFFFFFFFu;
        __syncthreads();
        for (int i = tid; i < len; i += 256) {
            uint64_t mag;
            int neg;
            scalar(vals, kind, base + i, mag, neg);
            const int d = (int)((mag >> (8 * w)) & 255);
            dig[i] = (uint8_t)d;
            sgn[i] = (uint8_t)neg;
            atomicAdd(&cnt[d], 1u);
        }
        __syncthreads();
        // counting sort by digit: perm[start(d) ..] holds the positions of digit d
        const uint32_t st = block_scan256(cnt[tid], sc, nullptr);
        cur[tid] = st;
        if (tid == 1) tot[0] = st;  // the start of digit 1: the number of zero digits
        __syncthreads();
        for (int i = tid; i < len; i += 256) perm[atomicAdd(&cur[dig[i]], 1u)] = (uint16_t)i;
        __syncthreads();
        // runs of the sorted list past the zero digits: thread t takes [r0, r1)
        const int skip = (int)tot[0], run = (len - skip + 255) / 256;
        const int r0 = skip + tid * run < len ? skip + tid * run : len;
        const int r1 = r0 + run < len ? r0 + run : len;
        uint32_t np = 0;  // partials of this run: its distinct digits
        for (int q = r0, prev = -1; q < r1; q++) {
            const int d = dig[perm[q]];
            if (d != prev) np++;
            prev = d;
        }
        const uint32_t off = block_scan256(np, sc, &tot[1]);
        {
            Jac acc = secp::jac_inf();
            int cd = -1;
            uint32_t k = off;
            for (int q = r0; q < r1; q++) {
                const int i = perm[q], d = dig[i];
                if (d != cd) {
                    if (cd >= 0) {
                        store_jac(pp[k], acc);
                        pd[k++] = (uint8_t)cd;
                    }
                    acc = secp::jac_inf();
                    cd = d;
                }
                Aff g;
                const uint32_t *gp = gens + 16 * (base + i);
                for (int l = 0; l < 8; l++) {
                    g.x.v[l] = gp[l];
                    g.y.v[l] = gp[8 + l];
                }
                if (sgn[i]) g.y = secp::fe_neg(g.y);
                acc = secp::jac_add_aff(acc, g);
            }
            if (cd >= 0) {
                store_jac(pp[k], acc);
                pd[k] = (uint8_t)cd;
            }
        }
        __syncthreads();
        // The partials are in digit order.  A digit spread over many runs (a
        // heavy bucket) has many partials: they are summed by a segmented tree,
        // each round adding to partial k the partial k + s of the same digit
        // (values read before any is written), until every segment's first
        // partial holds its sum.
        const uint32_t nparts = tot[1];
        if (tid == 0) tot[0] = 1;  // the longest segment
        for (uint32_t k = tid; k < nparts; k += 256) {
            if (k == 0 || pd[k] != pd[k - 1]) first[pd[k]] = k;
            atomicAdd(&cnt[pd[k]], 1u << 16);  // the partials of digit d, above cnt's 13-bit counts
        }
        __syncthreads();
        atomicMax(&tot[0], cnt[tid] >> 16);
        __syncthreads();
        for (uint32_t sd = 1; sd < tot[0]; sd <<= 1) {
            Jac add[2];
            bool has[2] = {false, false};
#pragma unroll
            for (int e = 0; e < 2; e++) {
                const uint32_t k = tid + 256 * e;
                if (k + sd < nparts && pd[k + sd] == pd[k]) {
                    add[e] = secp::jac_add(load_jac(pp[k]), load_jac(pp[k + sd]));
                    has[e] = true;
                }
            }
            __syncthreads();
#pragma unroll
            for (int e = 0; e < 2; e++)
                if (has[e]) store_jac(pp[tid + 256 * e], add[e]);
            __syncthreads();
        }
        if (tid >= 1 && first[tid] != 0xFFFFFFFFu) bucket = secp::jac_add(bucket, load_jac(pp[first[tid]]));
        __syncthreads();  // LDS reused by the next sort
    }
    if (tid >= 1) store_jac(out + (((size_t)w * gridDim.x + c) * 256 + tid) * kJacWords, bucket);
}

// Sums of 64 points per group of 64 threads (each thread's point in p[tid])
// by a tree in LDS; the group's first thread ends with the sum in p.
__device__ __forceinline__ void group64_tree(uint32_t (*p)[kJacWords])
{
    const int tid = threadIdx.x, j = tid & 63;
    for (int st = 32; st >= 1; st >>= 1) {
        __syncthreads();
        if (j < st) store_jac(p[tid], secp::jac_add(load_jac(p[tid]), load_jac(p[tid + st])));
    }
    __syncthreads();
}

// The tables of one batch: windows of table t are the global windows
// wpre[t] .. wpre[t + 1] - 1; its workspace starts off[t] bytes into ws:
// room for the chunks' bucket sums (W kMsmChunks 256 points, of which the
// bucket pass fills W C 256, window-major), the bucket sums S (W 256),
// their bit sums U (W 8).
struct MsmBatch {
    int count;
    uint32_t wpre[kCommitBatchMax + 1];
    uint32_t C[kCommitBatchMax];
    uint64_t off[kCommitBatchMax];
};
__device__ __forceinline__ int batch_table(const MsmBatch &b, uint32_t gw)
{
    int t = 0;
    while (t + 1 < b.count && gw >= b.wpre[t + 1]) t++;
    return t;
}
__device__ __forceinline__ uint32_t *batch_chunks(char *ws, const MsmBatch &b, int t)
{
    return (uint32_t *)(ws + b.off[t]);
}
__device__ __forceinline__ uint32_t *batch_S(char *ws, const MsmBatch &b, int t)
{
    const uint32_t W = b.wpre[t + 1] - b.wpre[t];
    return batch_chunks(ws, b, t) + (size_t)W * kMsmChunks * 256 * kJacWords;
}
__device__ __forceinline__ uint32_t *batch_U(char *ws, const MsmBatch &b, int t)
{
    const uint32_t W = b.wpre[t + 1] - b.wpre[t];
    return batch_S(ws, b, t) + (size_t)W * 256 * kJacWords;
}

// S[w][b] = sum over the C chunks of the chunks' bucket b of window w: 64
// threads per bucket, each a strided share, then a tree.  Four buckets of
// one window per workgroup; the workgroups run over the batch's windows.
__global__ __launch_bounds__(256) void k_pip_bucket_sums(char *ws, MsmBatch bt)
{
    __shared__ uint32_t part[256][kJacWords];
    const int tid = threadIdx.x, g = tid >> 6, j = tid & 63;
    const uint32_t wb = blockIdx.x * 4 + g, gw = wb >> 8, b = wb & 255;  // (global window, bucket)
    const int t = batch_table(bt, gw);                                     // workgroup-uniform
    const uint32_t w = gw - bt.wpre[t];
    const int C = (int)bt.C[t];
    const uint32_t *in = batch_chunks(ws, bt, t);
    Jac acc = secp::jac_inf();
    if (b >= 1)
        for (int c = j; c < C; c += 64) acc = secp::jac_add(acc, load_jac(in + (((size_t)w * C + c) * 256 + b) * kJacWords));
    store_jac(part[tid], acc);
    group64_tree(part);
    if (j == 0) store_jac(batch_S(ws, bt, t) + ((size_t)w * 256 + b) * kJacWords, load_jac(part[tid]));
}

// U[w][k] = sum over the b with bit k of S[w][b] (128 buckets): 64 threads
// per (w, k), two buckets each, then a tree.
__global__ __launch_bounds__(256) void k_pip_bit_sums(char *ws, MsmBatch bt)
{
    __shared__ uint32_t part[256][kJacWords];
    const int tid = threadIdx.x, g = tid >> 6, j = tid & 63;
    const uint32_t wk = blockIdx.x * 4 + g, gw = wk >> 3, k = wk & 7;
    const int t = batch_table(bt, gw);  // workgroup-uniform (four bits of one window)
    const uint32_t w = gw - bt.wpre[t];
    const uint32_t *S = batch_S(ws, bt, t);
    Jac acc = secp::jac_inf();
    for (int q = j; q < 128; q += 64) {  // the q-th b with bit k set
        const int b = ((q >> k) << (k + 1)) | (1 << k) | (q & ((1 << k) - 1));
        acc = secp::jac_add(acc, load_jac(S + ((size_t)w * 256 + b) * kJacWords));
    }
    store_jac(part[tid], acc);
    group64_tree(part);
    if (j == 0) store_jac(batch_U(ws, bt, t) + ((size_t)w * 8 + k) * kJacWords, load_jac(part[tid]));
}

// P = sum_w 2^(8w) T_w, T_w = sum_k 2^k U[w][k]: the windows' T_w by one
// thread each, then Horner over the windows; affine bytes to out + 64 t.
// One workgroup per table.
__global__ __launch_bounds__(64) void k_pip_final(char *ws, MsmBatch bt, uint8_t *__restrict__ out)
{
    __shared__ uint32_t T[8][kJacWords];
    const int tid = threadIdx.x, t = blockIdx.x;
    const int W = (int)(bt.wpre[t + 1] - bt.wpre[t]);
    const uint32_t *U = batch_U(ws, bt, t);
    if (tid < W) {
        Jac acc = secp::jac_inf();
        for (int k = 7; k >= 0; k--) {
            acc = secp::jac_dbl(acc);
            acc = secp::jac_add(acc, load_jac(U + ((size_t)tid * 8 + k) * kJacWords));
        }
        store_jac(T[tid], acc);
    }
    __syncthreads();
    if (tid == 0) {
        Jac p = secp::jac_inf();
        for (int w = W - 1; w >= 0; w--) {
            for (int q = 0; q < 8; q++) p = secp::jac_dbl(p);
            p = secp::jac_add(p, load_jac(T[w]));
        }
        uint8_t bytes[64];
        secp::jac_encode(p, bytes);
        for (int i = 0; i < 64; i++) out[64 * (size_t)t + i] = bytes[i];
    }
}

size_t msm_batch_offsets(const int *kinds, int count, size_t *offs)
{
    size_t o = 0;
    for (int t = 0; t < count; t++) {
        offs[t] = o;
        o += (msm_workspace_bytes(kinds[t]) + 255) & ~(size_t)255;
    }
    return o;
}

void launch_commit_batch(const void *const *vals, const int *kinds, const uint64_t *ns, int count,
                         const uint32_t *gens, void *ws, uint8_t *out, hipStream_t st)
{
    MsmBatch bt{};
    bt.count = count;
    size_t offs[kCommitBatchMax];
    msm_batch_offsets(kinds, count, offs);
    for (int t = 0; t < count; t++) {
        const int W = msm_windows(kinds[t]);
        const uint64_t n = ns[t], subs = (n + kPipSub - 1) / kPipSub;
        const int C = (int)(subs < (uint64_t)kMsmChunks ? (subs ? subs : 1) : kMsmChunks);
        const uint64_t per = ((n + C - 1) / C + kPipSub - 1) / kPipSub * kPipSub;  // whole sorts per chunk but the last
        bt.wpre[t + 1] = bt.wpre[t] + (uint32_t)W;
        bt.C[t] = (uint32_t)C;
        bt.off[t] = offs[t];
        hipLaunchKernelGGL(k_pip_buckets, dim3(C, W), dim3(256), 0, st, vals[t], kinds[t], n, gens, per,
                           (uint32_t *)((char *)ws + offs[t]));
    }
    const uint32_t nw = bt.wpre[count];
    hipLaunchKernelGGL(k_pip_bucket_sums, dim3(nw * 64), dim3(256), 0, st, (char *)ws, bt);
    hipLaunchKernelGGL(k_pip_bit_sums, dim3(nw * 2), dim3(256), 0, st, (char *)ws, bt);
    hipLaunchKernelGGL(k_pip_final, dim3(count), dim3(64), 0, st, (char *)ws, bt, out);
}

void launch_commit(const void *vals, int kind, uint64_t n, const uint32_t *gens, void *ws, uint8_t *out,
                   hipStream_t st)
{
    launch_commit_batch(&vals, &kind, &n, 1, gens, ws, out, st);
}

}  // namespace ra
