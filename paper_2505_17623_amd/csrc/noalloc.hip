// noalloc.hip -- ra_mle_bind_noalloc: the multilinear binding of ra_mle_bind
// for callers that cannot allocate device memory.  Its eq table and the
// partial sums of a row binding live in one fixed device array per GPU
// (`scratch` below); the point travels as a kernel argument, so the call
// makes no allocation and no copy.
#include <mutex>

#include "common.hpp"
#include "ra.h"

using namespace ra;

namespace {
constexpr uint64_t kP = 0x1FFFFFFFFFFFFFFFull;
constexpr size_t kScratchBytes = (size_t)RA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

// Each GPU holds its own copy of this array until the process ends.  In host
// code its name is not a device address: only the pointer returned by
// hipGetSymbolAddress (kept per device below) is passed to kernels.
static __device__ __align__(256) uint64_t scratch[kScratchBytes / 8];

std::mutex g_mu;
uint64_t *g_ptr[kMaxDevices] = {};

// The device address of this GPU's scratch array, looked up once per device
// with that device current (the caller's current device).
ra_status scratch_ptr(uint64_t **out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RA_E_HIP;
    if (dev < 0 || dev >= kMaxDevices) return RA_E_HIP;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return RA_E_HIP;
        g_ptr[dev] = (uint64_t *)p;
    }
    *out = g_ptr[dev];
    return RA_OK;
}

bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }
int log2u(uint64_t x)
{
    int l = 0;
    while ((1ull << l) < x) l++;
    return l;
}
size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }
}  // namespace

extern "C" ra_status ra_mle_bind_noalloc(const void *d_T, ra_dtype dtype, uint32_t rows, uint32_t cols, int bind_rows,
                                         const uint64_t *h_point, uint32_t point_len, uint64_t *d_out,
                                         void *hip_stream)
{
    if (!d_T || !d_out || !is_pow2(rows) || !is_pow2(cols)) return RA_E_INVAL;
    if (dtype != RA_I16 && dtype != RA_I32 && dtype != RA_I64 && dtype != RA_FIELD) return RA_E_INVAL;
    const int v = log2u(bind_rows ? rows : cols);
    if ((int)point_len != v || (v && !h_point)) return RA_E_INVAL;
    EqPoint pt{};
    pt.v = v;  // v <= 31: rows and cols are 32-bit powers of two
    for (int i = 0; i < v; i++) {
        if (h_point[i] >= kP) return RA_E_INVAL;
        pt.z[i] = h_point[i];
    }
    // scratch layout: eq table (2^v words), then a row binding's chunk sums
    const size_t eq_bytes = round256(((size_t)1 << v) * 8);
    const size_t part_bytes = bind_rows ? round256((size_t)bind_rows_chunks(rows, cols) * cols * 8) : 0;
    if (eq_bytes + part_bytes > kScratchBytes) return RA_E_SCRATCH;
    uint64_t *base = nullptr;
    const ra_status st = scratch_ptr(&base);
    if (st != RA_OK) return st;
    uint64_t *eq = base, *part = base + eq_bytes / 8;
    hipStream_t s = (hipStream_t)hip_stream;
    launch_eq_table_val(pt, eq, s);
    if (bind_rows)
        launch_bind_rows(d_T, dtype, rows, cols, eq, part, d_out, s);
    else
        launch_bind_cols(d_T, dtype, rows, cols, eq, d_out, s);
    if (hipGetLastError() != hipSuccess) return RA_E_HIP;
    return RA_OK;
}
