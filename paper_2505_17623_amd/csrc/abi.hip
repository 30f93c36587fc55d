// abi.hip -- host driver behind the C ABI of include/ra.h: context, device
// workspace, per-layer protocol state, and the orchestration of the kernels
// of witness.hip and sumcheck.hip for each entry point.
#include <algorithm>
#include <cstring>
#include <functional>
#include <new>
#include <vector>

#include "commit.hpp"
#include "common.hpp"
#include "ra.h"
#include "stream.hpp"
#include "xsetup.hpp"

using namespace ra;

namespace {
constexpr uint64_t kP = 0x1FFFFFFFFFFFFFFFull;

bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }
int log2u(uint64_t x)
{
    int l = 0;
    while ((1ull << l) < x) l++;
    return l;
}
}  // namespace

struct ra_ctx {
    int device = 0;
    hipStream_t stream = nullptr;  // the caller's stream: every call is ordered on it
    uint64_t *d_chal = nullptr;
    uint64_t n_chal = 0;   // challenges on the device
    uint64_t cursor = 0;   // challenges consumed
    bool seeded = false;   // challenges drawn from `seed` (more are drawn on demand)
    uint64_t seed = 0;
    // per-layer state between the three prover calls
    int phase = 0;  // 0: expects matmul, 1: expects witness, 2: expects range
    uint32_t n = 0, m = 0, k = 0;
    uint64_t *d_eq = nullptr;  // E1 (n words) then E2 (k words)
    uint64_t *d_acc = nullptr;  // row-binding accumulators of the fused front (zero between calls)
    size_t acc_cap = 0;
    uint64_t r12_off = 0;  // the layer's (r1, r2): offset in the challenge stream
    bool link_ok = false;  // a layer over F_p has just been proven: its a* may be linked (ra_link_prove)
    sha::Transcript *d_fs = nullptr;  // the Fiat-Shamir transcript (ra_ctx_create_fs), on the device
    size_t eq_cap = 0;
    WitParams *d_params = nullptr;
    char *d_wit = nullptr;  // the witness's per-workgroup partials (min/max, claims, range flags)
    ClaimsJob pend_claims{};  // a deferred witness call's last step, run by the range call's set-up
    // the next witness call as announced by ra_witness_plan (fused into the
    // product when `fused`, with `ntiles` partials)
    struct WitPlan {
        bool valid = false, fused = false;
        uint32_t s = 0, relu = 0, mode = 0;
        int32_t t = -1;
        int32_t *R = nullptr;
        uint16_t *Rm = nullptr;
        int32_t *Y = nullptr, *Z = nullptr;
        uint64_t *bits = nullptr;
        uint64_t bits_words = 0;
        uint32_t ntiles = 0;
    } plan;
    uint64_t *d_claims = nullptr;  // R~, Rm~, Y~, Z~ at (r1, r2)
    int s = 0, relu = 0, mode = 0, t = 0, P = 0;
    // kernel-group timing (ra_ctx_set_profiling)
    bool prof_on = false;
    std::vector<hipEvent_t> ev_pool;                   // free events
    std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> ev_pending;
    double prof_ms[32] = {};
    uint64_t prof_n[32] = {};
    // scratch
    char *ws = nullptr;
    size_t ws_cap = 0;
    uint64_t *h_stage = nullptr;  // pinned host memory the kernels write the calls' outputs to
    uint64_t *d_stage = nullptr;  // its device address
    size_t stage_cap = 0, stage_used = 0;
    // host outputs waiting for their staged words (written at once in
    // synchronous mode, at ra_ctx_sync in deferred mode)
    struct Pending {
        size_t off;
        std::function<ra_status(const uint64_t *)> fill;
    };
    std::vector<Pending> pending;
    bool deferred = false;
    ra_status deferred_err = 0;  // first error met while completing deferred outputs
};

#define RA_HIP(call)                                      \
    do {                                                  \
        if ((call) != hipSuccess) return RA_E_HIP;        \
    } while (0)

namespace {

ra_status drain(ra_ctx *c);

// Make `need` challenges past the cursor available on the device.  A seeded
// context draws the stream again from its seed into a larger buffer (after
// waiting for its stream, so no kernel still reads the old one); a context
// with given challenges has no more.
ra_status ensure_chal(ra_ctx *c, uint64_t need)
{
    if (c->cursor + need <= c->n_chal) return RA_OK;
    if (!c->seeded) return RA_E_SEED;
    const uint64_t want = std::max<uint64_t>({2 * c->n_chal, c->cursor + need, (uint64_t)1 << 16});
    std::vector<uint64_t> h(want);
    ra::ChallengeStream cs(c->seed);
    for (uint64_t i = 0; i < want; i++) h[i] = cs.next();
    const ra_status r = drain(c);
    if (r != RA_OK && c->deferred_err == RA_OK) c->deferred_err = r;
    uint64_t *d = nullptr;
    if (hipMalloc((void **)&d, want * 8) != hipSuccess) return RA_E_NOMEM;
    if (hipMemcpy(d, h.data(), want * 8, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(d);
        return RA_E_HIP;
    }
    if (c->d_chal) RA_HIP(hipFree(c->d_chal));
    c->d_chal = d;
    c->n_chal = want;
    return RA_OK;
}

// Bump allocator over the context workspace (256-byte aligned pieces).
struct Carve {
    size_t off = 0;
    template <typename T> size_t take(size_t count)
    {
        const size_t o = off;
        off += (count * sizeof(T) + 255) & ~(size_t)255;
        return o;
    }
};

// The witness partials: min / max (2 words), claims (4 words) and a range
// flag (4 bytes) per workgroup, for at most kMaxBlocks workgroups.
constexpr size_t kWitMinMax = 0, kWitClaims = 16 * kMaxBlocks, kWitFlags = kWitClaims + 32 * kMaxBlocks,
                 kWitBytes = kWitFlags + 4 * kMaxBlocks;

ra_status ensure_ws(ra_ctx *c, size_t bytes);

// The workspace of a proving call: the caller's (d_ws, at least `bytes`) or
// the context's own, grown on demand.
ra_status call_ws(ra_ctx *c, void *d_ws, size_t ws_bytes, size_t bytes, char **base)
{
    if (d_ws) {
        if (ws_bytes < bytes) return RA_E_BUFSIZE;
        *base = (char *)d_ws;
        return RA_OK;
    }
    const ra_status st = ensure_ws(c, bytes);
    *base = c->ws;
    return st;
}

ra_status ensure_ws(ra_ctx *c, size_t bytes)
{
    if (bytes <= c->ws_cap) return RA_OK;
    RA_HIP(hipStreamSynchronize(c->stream));
    if (c->ws) RA_HIP(hipFree(c->ws));
    c->ws = nullptr;
    c->ws_cap = 0;
    const size_t want = std::max(bytes + bytes / 4, (size_t)1 << 20);
    if (hipMalloc((void **)&c->ws, want) != hipSuccess) return RA_E_NOMEM;
    c->ws_cap = want;
    return RA_OK;
}

ra_status ensure_eq(ra_ctx *c, size_t words)
{
    if (words <= c->eq_cap) return RA_OK;
    RA_HIP(hipStreamSynchronize(c->stream));
    if (c->d_eq) RA_HIP(hipFree(c->d_eq));
    c->d_eq = nullptr;
    c->eq_cap = 0;
    if (hipMalloc((void **)&c->d_eq, words * 8) != hipSuccess) return RA_E_NOMEM;
    c->eq_cap = words;
    return RA_OK;
}

// Row-binding accumulators for m columns (2 m words).  They are zero between
// calls: the first reader of each word clears it.
ra_status ensure_acc(ra_ctx *c, size_t m)
{
    if (2 * m <= c->acc_cap) return RA_OK;
    RA_HIP(hipStreamSynchronize(c->stream));
    if (c->d_acc) RA_HIP(hipFree(c->d_acc));
    c->d_acc = nullptr;
    c->acc_cap = 0;
    if (hipMalloc((void **)&c->d_acc, 2 * m * 8) != hipSuccess) return RA_E_NOMEM;
    RA_HIP(hipMemset(c->d_acc, 0, 2 * m * 8));
    c->acc_cap = 2 * m;
    return RA_OK;
}

// Kernel groups timed with events when profiling is on.
enum Group {
    G_EQ = 0, G_GEMM, G_BIND_ROWS, G_BIND_COLS, G_MM_ROUNDS, G_MM_TAIL, G_WIT_MINMAX, G_WIT_RESCALE,
    G_RANGE_SETUP, G_RANGE_PLANE, G_RANGE_ROUNDS, G_RANGE_TAIL, G_FRONT, G_COUNT
};
const char *const kGroupName[G_COUNT] = {
    "eq_table", "gemm_mfma", "bind_rows", "bind_cols", "matmul_rounds", "matmul_tail", "witness_minmax",
    "witness_rescale", "range_setup", "range_plane", "range_rounds", "range_tail", "matmul_front"};

hipEvent_t take_event(ra_ctx *c)
{
    if (c->ev_pool.empty()) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
}

// Record an event pair around a launch group (no-op unless profiling).
struct Timed {
    ra_ctx *c;
    int g;
    hipStream_t s;
    hipEvent_t a = nullptr;
    Timed(ra_ctx *c_, int g_, hipStream_t s_ = nullptr) : c(c_), g(g_), s(s_ ? s_ : c_->stream)
    {
        if (c->prof_on && (a = take_event(c))) (void)hipEventRecord(a, s);
    }
    ~Timed()
    {
        if (!a) return;
        hipEvent_t b = take_event(c);
        if (!b) {
            c->ev_pool.push_back(a);
            return;
        }
        (void)hipEventRecord(b, s);
        c->ev_pending.push_back({g, {a, b}});
    }
};

void flush_profile(ra_ctx *c)
{
    for (auto &p : c->ev_pending) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, p.second.first, p.second.second) == hipSuccess) {
            c->prof_ms[p.first] += ms;
            c->prof_n[p.first] += 1;
        }
        c->ev_pool.push_back(p.second.first);
        c->ev_pool.push_back(p.second.second);
    }
    c->ev_pending.clear();
}

// Write every pending host output from its staged words (the stream has been
// synchronised).  Returns the first error a fill reports.
ra_status complete(ra_ctx *c)
{
    ra_status first = RA_OK;
    for (auto &p : c->pending) {
        const ra_status r = p.fill(c->h_stage + p.off);
        if (first == RA_OK) first = r;
    }
    c->pending.clear();
    c->stage_used = 0;
    flush_profile(c);
    return first;
}

// Wait for all enqueued work and complete the pending outputs.
ra_status drain(ra_ctx *c)
{
    if (c->pend_claims.nblk > 0) {  // a witness call's last step not yet taken by a range call
        launch_claims_final(c->pend_claims, c->stream);
        c->pend_claims.nblk = 0;
    }
    RA_HIP(hipStreamSynchronize(c->stream));
    return complete(c);
}

ra_status alloc_stage(ra_ctx *c, size_t words)
{
    if (c->h_stage) RA_HIP(hipHostFree(c->h_stage));
    c->h_stage = c->d_stage = nullptr;
    c->stage_cap = 0;
    if (hipHostMalloc((void **)&c->h_stage, words * 8, hipHostMallocMapped) != hipSuccess) return RA_E_NOMEM;
    RA_HIP(hipHostGetDevicePointer((void **)&c->d_stage, c->h_stage, 0));
    c->stage_cap = words;
    return RA_OK;
}

// Reserve `words` of pinned host memory for a call's outputs; the kernels
// write them there directly.  *off receives the offset (host: h_stage + off,
// device: d_stage + off).  Call before enqueueing the call's kernels.
ra_status stage_take(ra_ctx *c, size_t words, size_t *off)
{
    const size_t need = (words + 7) & ~(size_t)7;
    if (c->stage_used + need > c->stage_cap) {
        // grow to four times what is pending (a caller that keeps many calls
        // pending soon stops growing) once it has been written out
        const size_t want = std::max({4 * (c->stage_used + need), 2 * c->stage_cap, (size_t)4096});
        const ra_status r = drain(c);
        if (r != RA_OK && c->deferred_err == RA_OK) c->deferred_err = r;
        const ra_status a = alloc_stage(c, want);
        if (a != RA_OK) return a;
    }
    *off = c->stage_used;
    c->stage_used += need;
    return RA_OK;
}

// Register `fill` to turn the call's staged words (at `off`) into its host
// outputs.  Synchronous mode: waits, fills and returns the fill's status.
// Deferred mode: returns at once; ra_ctx_sync fills.
ra_status finish(ra_ctx *c, size_t off, std::function<ra_status(const uint64_t *)> fill)
{
    RA_HIP(hipGetLastError());
    c->pending.push_back({off, std::move(fill)});
    if (c->deferred) return RA_OK;
    const ra_status r = drain(c);
    if (r != RA_OK) return r;
    const ra_status d = c->deferred_err;
    c->deferred_err = RA_OK;
    return d;
}

// Plane count of the bit table for given s, t, relu (the rule of the witness
// kernel, Sec. III-A-2 and III-B): s + (t + 2) (1 + relu) planes, rounded up to
// a power of two.
ra_status plane_params(int s, int t, int relu, int *P, int *lP)
{
    if (s + t + 3 > 61) return RA_E_FIELD_TOO_SMALL;
    if (t > 29) return RA_E_NOT_IMPLEMENTED;  // R, Y, Z are int32
    const int Q = s + (t + 2) * (relu ? 2 : 1);
    int p = 1, l = 0;
    while (p < Q) {
        p <<= 1;
        l++;
    }
    if (l > kMaxPlaneLog) return RA_E_NOT_IMPLEMENTED;  // one bit word per output
    *P = p;
    *lP = l;
    return RA_OK;
}

constexpr int kPartStride = kMaxUnits * kPartWidth;  // words per partial-sum slot
static_assert((1 << kXTailLog) <= kMaxUnits && kMaxBlocks <= kMaxUnits, "partials must fit a slot");

int log2_tail() { return log2u(tail_capacity(0)); }

// One sum-check instance over tables of 2^v entries (in place): fused global
// launches while the table exceeds the LDS tail, then the tail, which also
// assembles every round.  Round j's width = D + 1 evaluations go to
// tr[ev_base + width j]; the tables' final values to finals[0..NT); with
// sum_out >= 0 the claimed sum to tr[sum_out].  With tail_out given, the
// tail is not launched: its arguments and jobs go to tail_out / jobs_out for
// a launch that carries it as extra workgroups.
void run_instance(ra_ctx *c, hipStream_t st, int kind, uint64_t *t0, uint64_t *t1, uint64_t *t2, int v,
                  const uint64_t *rho, uint64_t *tr, int ev_base, int width, uint64_t *finals, int sum_out,
                  uint64_t *part, int g_rounds, int g_tail, TailArgs *tail_out = nullptr, XJobs *jobs_out = nullptr,
                  uint64_t *acc0 = nullptr)
{
    const int cmax = fused_rounds_max(kind), lt = log2_tail();
    XJobs jobs{};
    jobs.part = part;
    jobs.stride = kPartStride;
    jobs.tr = tr;
    int j = 0, lS = v;
    while (lS > lt) {
        const int C = std::min(cmax, lS - lt);
        {
            Timed tm(c, g_rounds, st);
            launch_rounds(kind, C, t0, t1, t2, 1ull << lS, rho + j, nullptr, part + (size_t)jobs.nslot * kPartStride,
                          kPartStride, st, j == 0 ? acc0 : nullptr);
        }
        const int nb = round_blocks(1ull << (lS - C));
        for (int r = 0; r < C; r++)
            jobs.s[jobs.nslot++] =
                Slot{nb, width, ev_base + width * (j + r), SLOT_COPY, 0, (j + r == 0) ? sum_out : -1, -1};
        lS -= C;
        j += C;
    }
    const TailArgs ta{t0, t1, t2, v - j, rho + j, tr, ev_base, j, sum_out, finals,
                      finals ? finals + 1 : nullptr, finals ? finals + 2 : nullptr, j == 0 ? acc0 : nullptr};
    if (tail_out) {
        *tail_out = ta;
        *jobs_out = jobs;
        return;
    }
    Timed tm(c, g_tail, st);
    launch_tail(kind, ta, jobs, st);
}
// Workspace pieces of a matrix call.
struct MatmulLayout {
    size_t o_a, o_b, o_scr, o_part, o_gemm, bytes;
};
MatmulLayout matmul_layout(bool a_i32, uint32_t n, uint32_t m, uint32_t k)
{
    const int nslots = std::max(1, log2u(m));
    Carve cv;
    MatmulLayout l;
    l.o_a = cv.take<uint64_t>(m);
    l.o_b = cv.take<uint64_t>(m);
    l.o_scr = cv.take<uint64_t>((size_t)bind_rows_chunks(n, m) * m);
    l.o_part = cv.take<uint64_t>((size_t)nslots * kPartStride);
    l.o_gemm = cv.take<char>(gemm_workspace_bytes(a_i32, n, m, k));
    l.bytes = cv.off;
    return l;
}

// Workspace pieces and pass schedule of a range call over N outputs and 2^lP
// planes.  Rounds over x: register passes of kXFuseMax rounds while more
// than kXTailLog + kXBlockMax variables remain, then one pass of Bp rounds
// per workgroup in LDS, then the last pass (one workgroup).
struct RangeLayout {
    int L, nhs, reg, Bp, gtiles, gblocks;
    size_t o_cst, o_bx, o_d, o_s, o_hs, o_ls, o_kr, o_kz, o_wsh, o_part, o_gp, o_gs, bytes;
};
RangeLayout range_layout(uint64_t N, int lP, int relu)
{
    RangeLayout l;
    const int lN = log2u(N);
    l.L = std::min(lN, kXSplitLog);
    l.nhs = lN > l.L ? 1 << (lN - l.L) : 1;
    const int v = std::min(lN, kXTailLog), rem = lN - v;
    l.reg = 0;
    while (rem - l.reg > kXBlockMax) l.reg += kXFuseMax;
    l.Bp = rem - l.reg;
    l.gtiles = plane_gram_tiles(lP);
    l.gblocks = plane_gram_blocks(N, lP);
    const int nslots = std::max(lN, 1);
    Carve cv;
    l.o_cst = cv.take<uint64_t>(C_WORDS);
    l.o_bx = cv.take<uint64_t>(N);
    l.o_d = cv.take<uint64_t>(relu ? N : 1);
    l.o_s = cv.take<uint64_t>(relu ? N : 1);
    l.o_hs = cv.take<uint64_t>(l.nhs);
    l.o_ls = cv.take<uint64_t>(2ull << l.L);
    l.o_kr = cv.take<uint64_t>(lN + 1);
    l.o_kz = cv.take<uint64_t>(lN + 1);
    l.o_wsh = cv.take<uint64_t>(1ull << l.Bp);
    l.o_part = cv.take<uint64_t>((size_t)nslots * kPartStride);
    l.o_gp = cv.take<uint64_t>((size_t)l.gblocks * l.gtiles * kGramTileWords);
    l.o_gs = cv.take<uint64_t>(64 * 64);
    l.bytes = cv.off;
    return l;
}
// Workspace pieces of a layer proven over F_{p^2} (sized for P = 64), and
// the device transcript's word offsets: c0, a*, b* (0-5), the claims R~, Rm~,
// Y~, Z~ (6-13), the range instance's claimed sum (14-15), b~(sigma)
// (16-17), r_at, y_at (18-21), then the matrix rounds (6 words each), the
// range rounds (8 each, for up to 6 + log N) and the ReLU rounds (8 each).
constexpr int kF2TrFixed = 22;
struct Fp2Layout {
    size_t o_gemm, o_e1, o_e2, o_scr, o_a, o_b, o_eq, o_eqr, o_eqz, o_bx, o_d, o_s, o_sig, o_one, o_gp0, o_gp1, o_g,
        o_part, o_cpart, o_cst, o_tr, tr_words, o_fsch, o_dig0, o_dig1, o_root, o_err, bytes;
};
// leaves of the witness tables' Merkle tree (R, Rm, Y, Z int32 / uint16, the bit words)
uint64_t witness_leaves(uint64_t N)
{
    auto ch = [](uint64_t b) { return (b + 1023) / 1024; };
    return 3 * ch(4 * N) + ch(2 * N) + ch(8 * N);
}
Fp2Layout fp2_layout(bool a_i32, uint32_t n, uint32_t m, uint32_t k)
{
    const uint64_t N = (uint64_t)n * k, H = N > 1 ? N / 2 : 1;
    const int lm = log2u(m), lN = log2u(N);
    const int gt = plane_gram_tiles(kMaxPlaneLog), gb = plane_gram_blocks(N, kMaxPlaneLog);
    Carve cv;
    Fp2Layout l;
    l.o_gemm = cv.take<char>(gemm_workspace_bytes(a_i32, n, m, k));
    l.o_e1 = cv.take<uint64_t>(2 * (size_t)n);
    l.o_e2 = cv.take<uint64_t>(2 * (size_t)k);
    l.o_scr = cv.take<uint64_t>((size_t)bind_rows_chunks(n, m) * m);
    l.o_a = cv.take<uint64_t>(2 * (size_t)m);
    l.o_b = cv.take<uint64_t>(2 * (size_t)m);
    l.o_eq = cv.take<uint64_t>(2 * N);
    l.o_eqr = cv.take<uint64_t>(2 * H);
    l.o_eqz = cv.take<uint64_t>(2 * H);
    l.o_bx = cv.take<uint64_t>(2 * N);
    l.o_d = cv.take<uint64_t>(2 * H);
    l.o_s = cv.take<uint64_t>(2 * H);
    l.o_sig = cv.take<uint64_t>(2 * 64);
    l.o_one = cv.take<uint64_t>(2);
    l.o_gp0 = cv.take<uint64_t>((size_t)gb * gt * kGramTileWords);
    l.o_gp1 = cv.take<uint64_t>((size_t)gb * gt * kGramTileWords);
    l.o_g = cv.take<uint64_t>(2 * 4096);
    l.o_part = cv.take<uint64_t>((size_t)(lm + 2 * lN + 1) * kF2MaxBlocks * 8);
    l.o_cpart = cv.take<uint64_t>((size_t)kF2MaxBlocks * 8);
    l.o_cst = cv.take<uint64_t>(8);
    l.tr_words = kF2TrFixed + 6 * (size_t)lm + 8 * (size_t)(kMaxPlaneLog + lN) + 8 * (size_t)lN;
    l.o_tr = cv.take<uint64_t>(l.tr_words);
    // Fiat-Shamir: the layer's drawn challenges (pairs), the Merkle digests, the root, a status word
    l.o_fsch = cv.take<uint64_t>(2 * ((size_t)log2u(n) + log2u(k) + lm + 4 + 2 * kMaxPlaneLog + 2 * (size_t)lN));
    l.o_dig0 = cv.take<uint32_t>(8 * witness_leaves(N));
    l.o_dig1 = cv.take<uint32_t>(8 * ((witness_leaves(N) + 3) / 4));
    l.o_root = cv.take<uint8_t>(32);
    l.o_err = cv.take<uint32_t>(1);
    l.bytes = cv.off;
    return l;
}
}  // namespace

extern "C" {

ra_status ra_workspace_size_fp2(uint32_t n, uint32_t m, uint32_t k, size_t *bytes)
{
    if (!bytes || !is_pow2(n) || !is_pow2(m) || !is_pow2(k)) return RA_E_INVAL;
    if (m > kGemmMaxInner || (uint64_t)n * k > kRangeMaxN) return RA_E_NOT_IMPLEMENTED;
    *bytes = fp2_layout(true, n, m, k).bytes;
    return RA_OK;
}

ra_status ra_workspace_size(uint32_t n, uint32_t m, uint32_t k, uint32_t P, size_t *bytes)
{
    if (!bytes || !is_pow2(n) || !is_pow2(m) || !is_pow2(k) || !is_pow2(P)) return RA_E_INVAL;
    const uint64_t N = (uint64_t)n * k;
    const int lP = log2u(P);
    if (m > kGemmMaxInner || N > kRangeMaxN || lP > kMaxPlaneLog) return RA_E_NOT_IMPLEMENTED;
    *bytes = std::max(matmul_layout(true, n, m, k).bytes, range_layout(N, lP, 1).bytes);
    return RA_OK;
}

const char *ra_status_str(ra_status st)
{
    switch (st) {
    case RA_OK: return "ok";
    case RA_E_INVAL: return "invalid argument";
    case RA_E_UNSUPPORTED_PRIME: return "unsupported prime (only 2^61 - 1)";
    case RA_E_FIELD_TOO_SMALL: return "field too small: s + t + 3 > 61";
    case RA_E_RANGE: return "value range: the given t does not hold R";
    case RA_E_SEED: return "challenge stream: seed 0, given challenges exhausted, or a challenge >= p";
    case RA_E_HIP: return "HIP runtime error";
    case RA_E_STATE: return "call out of the per-layer order";
    case RA_E_BUFSIZE: return "buffer too small";
    case RA_E_NOT_IMPLEMENTED: return "beyond this GPU path's limits (m <= 32768, s <= 16, t <= 29, P <= 64, N <= 2^31)";
    case RA_E_NOMEM: return "allocation failed";
    case RA_E_SCRATCH: return "needs more than the fixed scratch of ra_mle_bind_noalloc";
    default: return "unknown status";
    }
}

}  // extern "C"

namespace {
// A context with its fixed device buffers and `n` challenges from h (seeded:
// h is the stream's first n draws).
ra_status ctx_create(uint64_t p, const uint64_t *h, uint64_t n, bool seeded, uint64_t seed, void *hip_stream,
                     ra_ctx **out)
{
    ra_ctx *c = new (std::nothrow) ra_ctx();
    if (!c) return RA_E_NOMEM;
    (void)p;
    c->stream = (hipStream_t)hip_stream;
    c->seeded = seeded;
    c->seed = seed;
    ra_status st = RA_OK;
    if (hipGetDevice(&c->device) != hipSuccess) st = RA_E_HIP;
    if (st == RA_OK && hipMalloc((void **)&c->d_chal, std::max<uint64_t>(n, 1) * 8) != hipSuccess) st = RA_E_NOMEM;
    if (st == RA_OK && n && hipMemcpy(c->d_chal, h, n * 8, hipMemcpyHostToDevice) != hipSuccess) st = RA_E_HIP;
    static_assert(sizeof(WitParams) <= 64, "parameters precede the claims");
    if (st == RA_OK && hipMalloc((void **)&c->d_params, 128) != hipSuccess) st = RA_E_NOMEM;
    if (st == RA_OK && hipMalloc((void **)&c->d_wit, kWitBytes) != hipSuccess) st = RA_E_NOMEM;
    if (st == RA_OK) c->d_claims = (uint64_t *)((char *)c->d_params + 64);
    if (st == RA_OK) st = alloc_stage(c, 4096);
    if (st != RA_OK) {
        ra_ctx_destroy(c);
        return st;
    }
    c->n_chal = n;
    init_kernel_attributes();
    *out = c;
    return RA_OK;
}
}  // namespace

extern "C" {

ra_status ra_ctx_create(uint64_t p, uint64_t seed, void *hip_stream, ra_ctx **out)
{
    if (!out) return RA_E_INVAL;
    *out = nullptr;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    if (seed == 0) return RA_E_SEED;
    const uint64_t n = 1ull << 16;  // first draws; more on demand (ensure_chal)
    std::vector<uint64_t> h(n);
    ra::ChallengeStream cs(seed);
    for (uint64_t i = 0; i < n; i++) h[i] = cs.next();
    return ctx_create(p, h.data(), n, true, seed, hip_stream, out);
}

ra_status ra_ctx_create_stream(uint64_t p, const uint64_t *h_challenges, uint64_t n_challenges, void *hip_stream,
                               ra_ctx **out)
{
    if (!out) return RA_E_INVAL;
    *out = nullptr;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    if (n_challenges && !h_challenges) return RA_E_INVAL;
    for (uint64_t i = 0; i < n_challenges; i++)
        if (h_challenges[i] >= kP) return RA_E_SEED;
    return ctx_create(p, h_challenges, n_challenges, false, 0, hip_stream, out);
}

ra_status ra_ctx_create_fs(uint64_t p, const uint8_t *domain, void *hip_stream, ra_ctx **out)
{
    if (!out || !domain) return RA_E_INVAL;
    *out = nullptr;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    ra_ctx *c = nullptr;
    ra_status st = ctx_create(p, nullptr, 0, false, 0, hip_stream, &c);
    if (st != RA_OK) return st;
    sha::Transcript t;
    sha::fs_init(t, domain);
    if (hipMalloc((void **)&c->d_fs, sizeof(sha::Transcript)) != hipSuccess) st = RA_E_NOMEM;
    if (st == RA_OK && hipMemcpy(c->d_fs, &t, sizeof(t), hipMemcpyHostToDevice) != hipSuccess) st = RA_E_HIP;
    if (st != RA_OK) {
        ra_ctx_destroy(c);
        return st;
    }
    *out = c;
    return RA_OK;
}

ra_status ra_ctx_destroy(ra_ctx *c)
{
    if (!c) return RA_E_INVAL;
    if (c->stream || c->ws || c->d_chal) (void)hipStreamSynchronize(c->stream);
    if (c->d_chal) (void)hipFree(c->d_chal);
    if (c->d_fs) (void)hipFree(c->d_fs);
    if (c->d_eq) (void)hipFree(c->d_eq);
    if (c->d_acc) (void)hipFree(c->d_acc);
    if (c->d_params) (void)hipFree(c->d_params);
    if (c->d_wit) (void)hipFree(c->d_wit);
    if (c->ws) (void)hipFree(c->ws);
    if (c->h_stage) (void)hipHostFree(c->h_stage);
    flush_profile(c);
    for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
    delete c;
    return RA_OK;
}

ra_status ra_ctx_cursor(const ra_ctx *c, uint64_t *consumed)
{
    if (!c || !consumed) return RA_E_INVAL;
    *consumed = c->cursor;
    return RA_OK;
}

ra_status ra_ctx_set_deferred(ra_ctx *c, int on)
{
    if (!c) return RA_E_INVAL;
    if (!on && c->deferred) {
        const ra_status r = drain(c);
        if (r != RA_OK && c->deferred_err == RA_OK) c->deferred_err = r;
    }
    c->deferred = on != 0;
    return RA_OK;
}

ra_status ra_ctx_sync(ra_ctx *c)
{
    if (!c) return RA_E_INVAL;
    const ra_status r = drain(c);
    ra_status first = c->deferred_err != RA_OK ? c->deferred_err : r;
    c->deferred_err = RA_OK;
    return first;
}

ra_status ra_ctx_set_profiling(ra_ctx *c, int on)
{
    if (!c) return RA_E_INVAL;
    {
        const ra_status r = drain(c);
        if (r != RA_OK && c->deferred_err == RA_OK) c->deferred_err = r;
    }
    c->prof_on = on != 0;
    for (int g = 0; g < G_COUNT; g++) {
        c->prof_ms[g] = 0;
        c->prof_n[g] = 0;
    }
    return RA_OK;
}

ra_status ra_ctx_profile(const ra_ctx *c, uint32_t index, const char **name, double *total_ms, uint64_t *launches)
{
    if (!c || index >= (uint32_t)G_COUNT) return RA_E_INVAL;
    if (name) *name = kGroupName[index];
    if (total_ms) *total_ms = c->prof_ms[index];
    if (launches) *launches = c->prof_n[index];
    return RA_OK;
}

ra_status ra_mle_bind(ra_ctx *c, const void *d_T, ra_dtype dtype, uint32_t rows, uint32_t cols, int bind_rows,
                      const uint64_t *h_point, uint32_t point_len, uint64_t *d_out)
{
    if (!c || !d_T || !d_out || !is_pow2(rows) || !is_pow2(cols)) return RA_E_INVAL;
    if (dtype != RA_I16 && dtype != RA_I32 && dtype != RA_I64 && dtype != RA_FIELD) return RA_E_INVAL;
    const int v = log2u(bind_rows ? rows : cols);
    if ((int)point_len != v || (v && !h_point)) return RA_E_INVAL;
    for (int i = 0; i < v; i++)
        if (h_point[i] >= kP) return RA_E_INVAL;
    Carve cv;
    const size_t o_pt = cv.take<uint64_t>(std::max(v, 1));
    const size_t o_eq = cv.take<uint64_t>(1ull << v);
    const size_t o_scr = cv.take<uint64_t>(bind_rows ? (size_t)bind_rows_chunks(rows, cols) * cols : 1);
    ra_status st = ensure_ws(c, cv.off);
    if (st != RA_OK) return st;
    uint64_t *pt = (uint64_t *)(c->ws + o_pt), *eq = (uint64_t *)(c->ws + o_eq), *scr = (uint64_t *)(c->ws + o_scr);
    // a synchronous utility: land any deferred outputs, then use the staging area for the point
    st = drain(c);
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    if ((size_t)v > c->stage_cap) return RA_E_INVAL;  // log2 of a 32-bit dimension
    if (v) std::memcpy(c->h_stage, h_point, (size_t)v * 8);
    RA_HIP(hipMemcpyAsync(pt, c->h_stage, (size_t)std::max(v, 1) * 8, hipMemcpyHostToDevice, c->stream));
    launch_eq_table(pt, v, eq, c->stream);
    if (bind_rows)
        launch_bind_rows(d_T, dtype, rows, cols, eq, scr, d_out, c->stream);
    else
        launch_bind_cols(d_T, dtype, rows, cols, eq, d_out, c->stream);
    RA_HIP(hipGetLastError());
    RA_HIP(hipStreamSynchronize(c->stream));
    return RA_OK;
}

ra_status ra_sumcheck_matmul_prove(ra_ctx *c, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                                   uint32_t m, uint32_t k, int64_t *d_C, void *d_ws, size_t ws_bytes,
                                   ra_matmul_proof *out)
{
    if (!c || !d_A || !d_B || !d_C || !out) return RA_E_INVAL;
    if (!is_pow2(n) || !is_pow2(m) || !is_pow2(k)) return RA_E_INVAL;
    if (a_dtype != RA_I16 && a_dtype != RA_I32) return RA_E_INVAL;
    if (m > kGemmMaxInner) return RA_E_NOT_IMPLEMENTED;  // exactness of the limb products
    if ((uint64_t)n * k > kRangeMaxN) return RA_E_NOT_IMPLEMENTED;  // the layer's range call could not run
    if (c->phase != 0) return RA_E_STATE;
    const int ln = log2u(n), lm = log2u(m), lk = log2u(k);
    if (lm && !out->evals) return RA_E_INVAL;
    const uint64_t need = (uint64_t)ln + lk + lm;
    ra_status st = ensure_chal(c, need);
    if (st != RA_OK) return st;
    const uint64_t *r1 = c->d_chal + c->cursor, *r2 = r1 + ln, *rho = r2 + lk;

    if ((st = ensure_eq(c, (size_t)n + k)) != RA_OK) return st;
    const size_t trw = 3 + 3 * (size_t)lm;
    const MatmulLayout ml = matmul_layout(a_dtype == RA_I32, n, m, k);
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, ml.bytes, &ws)) != RA_OK) return st;
    const size_t o_gemm = ml.o_gemm;
    uint64_t *a = (uint64_t *)(ws + ml.o_a), *b = (uint64_t *)(ws + ml.o_b);
    size_t o_tr = 0;
    if ((st = stage_take(c, trw, &o_tr)) != RA_OK) return st;
    uint64_t *scr = (uint64_t *)(ws + ml.o_scr), *part = (uint64_t *)(ws + ml.o_part), *tr = c->d_stage + o_tr;
    uint64_t *E1 = c->d_eq, *E2 = c->d_eq + n;
    hipStream_t s = c->stream;

    // the sum-check chain (eq tables, bindings, rounds), then the product C,
    // all on the caller's stream
    hipStream_t z = s;
    // The fused front (one launch: limb split, both bindings, eq tables) where
    // the shapes allow; else eq tables, row binding, column binding.
    const bool fused = front_supported(a_dtype == RA_I32, n, m, k, d_A, d_B);
    if (fused) {
        if ((st = ensure_acc(c, m)) != RA_OK) return st;
        Timed tm(c, G_FRONT, z);
        launch_front(d_A, a_dtype == RA_I32, d_B, n, m, k, r1, ln, r2, lk, c->d_acc, b, E1, E2, ws + o_gemm, z);
    } else {
        {
            Timed tm(c, G_EQ, z);
            launch_eq_tables(r1, ln, E1, r2, lk, E2, z);
        }
        ChunkSum cs{};
        {
            Timed tm(c, G_BIND_ROWS, z);
            cs = launch_bind_rows_chunks(d_A, a_dtype, n, m, E1, scr, a, z);
        }
        {   // B bound on its columns; extra workgroups finish the row binding of A
            Timed tm(c, G_BIND_COLS, z);
            launch_bind_cols(d_B, RA_I16, m, k, E2, b, z, &cs);
        }
    }
    // transcript: [c0][evals 3 lm][a*][b*]; the instance's tail runs as extra
    // workgroups of the product launch
    TailArgs ta{};
    XJobs tjobs{};
    run_instance(c, z, KIND_MATMUL, a, b, nullptr, lm, rho, tr, 1, 3, tr + 1 + 3 * lm, 0, part, G_MM_ROUNDS,
                 G_MM_TAIL, &ta, &tjobs, fused ? c->d_acc : nullptr);
    // an announced witness (ra_witness_plan) runs in the product's epilogue
    // when every output tile has a partial slot
    WitEpi we{};
    bool fuse_w = false;
    if (c->plan.valid) {
        const uint32_t nt = gemm_tiles(n, k);
        fuse_w = nt <= (uint32_t)kMaxBlocks && c->plan.bits_words >= (uint64_t)n * k;
        if (fuse_w) {
            const auto &pl = c->plan;
            we = WitEpi{(int)pl.s, pl.t, (int)pl.relu, pl.mode == RA_ROUND_NEAREST ? (int64_t)1 << (pl.s - 1) : 0,
                        E1, E2, pl.R, pl.Rm, pl.Y, pl.Z, pl.bits, (uint64_t *)(c->d_wit + kWitClaims),
                        (uint32_t *)(c->d_wit + kWitFlags)};
            c->plan.ntiles = nt;
        }
        c->plan.fused = fuse_w;
    }
    {
        Timed tm(c, G_GEMM);
        launch_gemm_mfma(d_A, a_dtype == RA_I32, d_B, d_C, n, m, k, ws + o_gemm, s, &ta, &tjobs, fused,
                         fuse_w ? &we : nullptr);
    }
    c->n = n;
    c->m = m;
    c->k = k;
    c->r12_off = c->cursor;
    c->phase = 1;
    c->link_ok = false;
    c->cursor += need;
    return finish(c, o_tr, [out, lm](const uint64_t *h) {
        out->log_m = (uint32_t)lm;
        out->c0 = h[0];
        if (lm) std::memcpy(out->evals, h + 1, 3 * (size_t)lm * 8);
        out->a_star = h[1 + 3 * lm];
        out->b_star = h[2 + 3 * lm];
        return (ra_status)RA_OK;
    });
}

ra_status ra_witness_plan(ra_ctx *c, uint32_t s, uint32_t relu, uint32_t round_mode, int32_t t, int32_t *d_R,
                          uint16_t *d_Rm, int32_t *d_Y, int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words)
{
    if (!c || !d_R || !d_Rm || !d_Y || !d_Z || !d_bits) return RA_E_INVAL;
    if (c->phase != 0) return RA_E_STATE;
    if (s < 1 || relu > 1 || round_mode > 1 || t < 0) return RA_E_INVAL;
    if (s > 16) return RA_E_NOT_IMPLEMENTED;  // Rm is uint16
    int P = 0, lP = 0;
    const ra_status pst = plane_params((int)s, t, (int)relu, &P, &lP);
    if (pst != RA_OK) return pst;
    auto &pl = c->plan;
    pl.valid = true;
    pl.fused = false;
    pl.s = s;
    pl.relu = relu;
    pl.mode = round_mode;
    pl.t = t;
    pl.R = d_R;
    pl.Rm = d_Rm;
    pl.Y = d_Y;
    pl.Z = d_Z;
    pl.bits = d_bits;
    pl.bits_words = bits_words;
    pl.ntiles = 0;
    return RA_OK;
}

ra_status ra_rescale_relu_witness(ra_ctx *c, const int64_t *d_C, uint32_t n, uint32_t k, int32_t *d_R,
                                  uint16_t *d_Rm, int32_t *d_Y, int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words,
                                  void *d_ws, size_t ws_bytes, ra_witness_info *io)
{
    (void)d_ws;  // the witness keeps its partials in the context (a deferred
    (void)ws_bytes;  // call's last step runs in the next call)
    if (!c || !d_C || !d_R || !d_Rm || !d_Y || !d_Z || !d_bits || !io) return RA_E_INVAL;
    if (c->phase != 1) return RA_E_STATE;
    if (n != c->n || k != c->k) return RA_E_INVAL;
    if (io->s < 1 || io->relu > 1 || io->round_mode > 1 || io->t < -1) return RA_E_INVAL;
    if (io->s > 16) return RA_E_NOT_IMPLEMENTED;  // Rm is uint16
    const uint64_t N = (uint64_t)n * k;
    if (bits_words < N) return RA_E_BUFSIZE;
    // with t given and deferred outputs, the plane count is known on the host
    // and the call need not wait; otherwise it waits for t and P
    // with t given, the parameters (but for the range check of R, which the
    // rescale pass makes) are fixed on the host; in deferred mode the call
    // then need not wait.  Otherwise a min / max pass finds t and P first.
    int hP = 0, hlP = 0;
    const bool given = io->t >= 0, known = c->deferred && given;
    WitParams hp{};
    if (given) {
        const ra_status pst = plane_params((int)io->s, io->t, (int)io->relu, &hP, &hlP);
        if (pst != RA_OK) return pst;
        hp.status = 0;
        hp.t = io->t;
        hp.P = hP;
        hp.lP = hlP;
        hp.s = (int)io->s;
        hp.relu = (int)io->relu;
        hp.mode = (int)io->round_mode;
        hp.t_in = io->t;
    }
    static_assert(kMaxBlocks >= 1, "witness partials");  // witness_blocks(N) <= kMaxBlocks
    ra_status st = RA_OK;
    const int lk = log2u(k);
    size_t o_st = 0;
    if ((st = stage_take(c, 12, &o_st)) != RA_OK) return st;
    // the product's epilogue made the outputs and per-tile partials if this
    // call is the one announced; the plan is spent either way
    const auto pl = c->plan;
    c->plan.valid = c->plan.fused = false;
    const bool planned = pl.valid && pl.fused && given && io->s == pl.s && io->relu == pl.relu &&
                         io->round_mode == pl.mode && io->t == pl.t && d_R == pl.R && d_Rm == pl.Rm && d_Y == pl.Y &&
                         d_Z == pl.Z && d_bits == pl.bits;
    if (planned) {
        const ClaimsJob j{(const uint64_t *)(c->d_wit + kWitClaims), (int)pl.ntiles, c->d_params, c->d_claims,
                          c->d_stage + o_st, hp, 1, (const uint32_t *)(c->d_wit + kWitFlags)};
        if (known) {
            c->pend_claims = j;
        } else {
            Timed tm(c, G_WIT_RESCALE);
            launch_claims_final(j, c->stream);
        }
    }
    if (!given) {
        Timed tm(c, G_WIT_MINMAX);
        launch_witness_params(d_C, N, (int)io->s, (int)io->relu, (int)io->round_mode, io->t,
                              (int64_t *)(c->d_wit + kWitMinMax), c->d_params, c->stream);
    }
    if (!planned) {   // A call that does not wait (deferred, t given) leaves its last step, the
        // sum of the claims, to the range call that must follow (its set-up
        // launch), or to the next wait on the context.
        Timed tm(c, G_WIT_RESCALE);
        launch_witness_rescale(d_C, N, lk, c->d_eq, c->d_eq + n, d_R, d_Rm, d_Y, d_Z, d_bits,
                               (uint64_t *)(c->d_wit + kWitClaims), c->d_params, c->d_claims, c->d_stage + o_st,
                               c->stream, given ? &hp : nullptr, (uint32_t *)(c->d_wit + kWitFlags),
                               known ? &c->pend_claims : nullptr);
    }
    // parameters (words 0-7) and claims (words 8-11) are staged together
    auto fill = [c, io, known](const uint64_t *h) {
        WitParams prm;
        std::memcpy(&prm, h, sizeof(prm));
        if (prm.status != 0) return (ra_status)prm.status;
        io->t = prm.t;
        io->P = (uint32_t)prm.P;
        io->r_claim = h[8];
        io->rm_claim = h[9];
        io->y_claim = h[10];
        io->z_claim = h[11];
        if (!known) {  // the layer state advances once t and P are known
            c->s = (int)io->s;
            c->relu = (int)io->relu;
            c->mode = (int)io->round_mode;
            c->t = prm.t;
            c->P = prm.P;
            c->phase = 2;
        }
        return (ra_status)RA_OK;
    };
    if (known) {
        c->s = (int)io->s;
        c->relu = (int)io->relu;
        c->mode = (int)io->round_mode;
        c->t = io->t;
        c->P = hP;
        c->phase = 2;
        io->P = (uint32_t)hP;
        return finish(c, o_st, fill);
    }
    const bool was = c->deferred;
    c->deferred = false;  // this call must wait for t and P
    st = finish(c, o_st, fill);
    c->deferred = was;
    return st;
}

ra_status ra_range_prove(ra_ctx *c, const uint64_t *d_bits, const int32_t *d_R, const int32_t *d_Y, uint32_t n,
                         uint32_t k, const ra_witness_info *info, void *d_ws, size_t ws_bytes, ra_range_proof *out)
{
    if (!c || !d_bits || !info || !out || !out->evals) return RA_E_INVAL;
    if (c->phase != 2) return RA_E_STATE;
    if (n != c->n || k != c->k) return RA_E_INVAL;
    if ((int)info->s != c->s || (int)info->relu != c->relu || (int)info->round_mode != c->mode || info->t != c->t ||
        (int)info->P != c->P)
        return RA_E_INVAL;
    const int relu = c->relu;
    if (relu && (!d_R || !d_Y || !out->relu_evals)) return RA_E_INVAL;
    const uint64_t N = (uint64_t)n * k;
    const int lP = log2u((uint64_t)c->P), lN = log2u(N), lk = log2u(k), R = lP + lN;
    if (N > kRangeMaxN) return RA_E_NOT_IMPLEMENTED;  // exact int32 sums of the plane rounds
    const uint64_t need = 4 + (uint64_t)lP + R + (relu ? lN : 0);
    ra_status st = ensure_chal(c, need);
    if (st != RA_OK) return st;
    const uint64_t *lam = c->d_chal + c->cursor, *sigma = lam + 4 + lP, *rho2 = sigma + R;
    const uint64_t *d_r12 = c->d_chal + c->r12_off;

    const RangeLayout rl = range_layout(N, lP, relu);
    const int L = rl.L, nhs = rl.nhs, reg = rl.reg, Bp = rl.Bp;
    // planes the witness writes (the bit words are zero above them): the Gram
    // pass skips a block of sixteen planes that holds none
    const int pused = c->s + (c->t + 2) * (relu ? 2 : 1);
    const int gtiles = plane_gram_tiles(lP, pused), gblocks = rl.gblocks;  // workspace sized for rl.gtiles >= gtiles
    // transcript: [evals 4R][(unused)][bits_claim][range_sum][relu evals 4 lN][(unused)][r_at][y_at]
    const size_t F_R = 4 * (size_t)R, RS = F_R + 2, Z0 = F_R + 3, FZ = Z0 + 4 * (size_t)lN, trw = FZ + 3;
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, rl.bytes, &ws)) != RA_OK) return st;
    uint64_t *cst = (uint64_t *)(ws + rl.o_cst), *Bx = (uint64_t *)(ws + rl.o_bx);
    uint64_t *D = (uint64_t *)(ws + rl.o_d), *S = (uint64_t *)(ws + rl.o_s);
    uint64_t *HS = (uint64_t *)(ws + rl.o_hs), *LS = (uint64_t *)(ws + rl.o_ls);
    uint64_t *Kr = (uint64_t *)(ws + rl.o_kr), *Kz = (uint64_t *)(ws + rl.o_kz);
    uint64_t *WSh = (uint64_t *)(ws + rl.o_wsh);
    size_t o_tr = 0;
    if ((st = stage_take(c, trw, &o_tr)) != RA_OK) return st;
    uint64_t *part = (uint64_t *)(ws + rl.o_part), *tr = c->d_stage + o_tr;
    uint64_t *gpart = (uint64_t *)(ws + rl.o_gp), *gsum = (uint64_t *)(ws + rl.o_gs);
    const uint64_t *sigx = sigma + lP, *rz = relu ? rho2 : nullptr;
    hipStream_t s = c->stream;

    // With a register pass (reg > 0) the set-up of the rounds over x runs in
    // the Gram pass (its consumer waves, while the first slab is built) and
    // the Gram reduction, the constant block and a deferred witness step ride
    // in the register pass's launch; the plane rounds are then evaluated one
    // launch later.  Otherwise a launch of its own runs all of that between
    // the Gram pass and the first x launch.
    const XSetupArgs xs{d_r12, sigx, rz, lN, L, nhs, HS, LS, Kr, Kz, WSh, reg, Bp};
    const bool riding = reg > 0 && x_setup_count(xs) <= plane_gram_set_up_threads(N, lP);
    const RangeConsts rc{lam, c->d_params, c->d_claims, lP, cst, tr + RS, c->pend_claims};
    c->pend_claims.nblk = 0;  // taken by this call's launches
    const RangeRiders riders{gpart, gblocks, gtiles, gram_reduce_groups(gtiles), gsum, rc};
    {   // plane rounds: Gram matrix on the matrix cores, Bx per output
        Timed tm(c, G_RANGE_PLANE);
        launch_plane_gram(lP, d_bits, N, lk, c->d_eq, c->d_eq + n, sigma, Bx, gpart, riding ? &xs : nullptr, s,
                          nullptr, pused);
    }
    if (!riding) {  // the Gram matrix; further workgroups: the constant block and the x set-up
        Timed tm(c, G_RANGE_SETUP);
        launch_gram_reduce(lP, N, gpart, gsum, rc, xs, s, pused);
    }
    // Each x launch's extra workgroups assemble the rounds of the launch
    // before it; the first one also evaluates the plane rounds (the second
    // one when the Gram reduction rides in the first), the last assembles
    // its own.
    const XConst xc{cst + C_EP, d_r12, Kr, Kz};
    XJobs jobs{};
    jobs.nplane = riding ? 0 : lP;
    jobs.stride = kPartStride;
    jobs.tr = tr;
    jobs.xc = xc;
    jobs.pa = PlaneArgs{gsum, sigma, cst, tr, lP};
    auto next_jobs = [&](int j0, int nr, int units) {
        jobs.nplane = riding && j0 == 0 ? lP : 0;
        jobs.nslot = nr;
        jobs.part = part + (size_t)j0 * kPartStride;
        for (int r = 0; r < nr; r++)
            jobs.s[r] = Slot{units, kPartWidth, 4 * (lP + j0 + r), SLOT_X, j0 + r, -1,
                             relu ? (int)Z0 + 4 * (j0 + r) : -1};
    };
    int j = 0, lS = lN;
    for (; j < reg; j += kXFuseMax, lS -= kXFuseMax) {
        const XArgs xa{Bx, D, S, d_R, d_Y, HS, LS, d_r12, sigx + j, rz ? rz + j : nullptr,
                       part + (size_t)j * kPartStride, lN, L, j};
        {
            Timed tm(c, G_RANGE_ROUNDS);
            launch_xrounds(kXFuseMax, j == 0, relu != 0, xa, 1ull << lS, kPartStride, jobs, s,
                           riding && j == 0 ? &riders : nullptr);
        }
        next_jobs(j, kXFuseMax, xround_units(1ull << (lS - kXFuseMax), relu != 0));
    }
    XBlockArgs xb{Bx, D, S, d_R, d_Y, HS, LS, d_r12, WSh, nullptr, nullptr, nullptr, kPartStride, lN, L, 0, 0, 0,
                  tr, 0, 0, tr + F_R + 1, tr + FZ + 1, tr + FZ + 2, xc};
    if (Bp > 0) {
        xb.rho_a = sigx + j;
        xb.rho_z = rz ? rz + j : nullptr;
        xb.part = part + (size_t)j * kPartStride;
        xb.j = j;
        xb.B = Bp;
        xb.lS = lS;
        {
            Timed tm(c, G_RANGE_ROUNDS);
            launch_xblock(relu != 0, j == 0, xb, jobs, s);
        }
        next_jobs(j, Bp, 1 << (lS - Bp));
        j += Bp;
        lS -= Bp;
    }
    xb.W = LS;  // the last pass's window r_{j+1 .. lN-1} ends at the last variable
    xb.rho_a = sigx + j;
    xb.rho_z = rz ? rz + j : nullptr;
    xb.j = j;
    xb.B = lS;
    xb.lS = lS;
    xb.out0 = 4 * (lP + j);
    xb.out2 = relu ? (int)Z0 + 4 * j : -1;
    {
        Timed tm(c, G_RANGE_TAIL);
        launch_xblock(relu != 0, j == 0, xb, jobs, s);
    }
    c->phase = 0;
    c->link_ok = true;
    c->cursor += need;
    return finish(c, o_tr, [out, R, relu, lN, F_R, RS, Z0, FZ](const uint64_t *h) {
        out->rounds = (uint32_t)R;
        std::memcpy(out->evals, h, 4 * (size_t)R * 8);
        out->bits_claim = h[F_R + 1];
        out->range_sum = h[RS];
        out->relu_rounds = relu ? (uint32_t)lN : 0;
        if (relu) {
            if (lN) std::memcpy(out->relu_evals, h + Z0, 4 * (size_t)lN * 8);
            out->r_at = h[FZ + 1];
            out->y_at = h[FZ + 2];
        } else {
            out->r_at = out->y_at = 0;
        }
        return (ra_status)RA_OK;
    });
}

ra_status ra_prove_layer_fp2(ra_ctx *c, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                             uint32_t m, uint32_t k, int64_t *d_C, int32_t *d_R, uint16_t *d_Rm, int32_t *d_Y,
                             int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words, void *d_ws, size_t ws_bytes,
                             ra_layer_proof_fp2 *io)
{
    if (!c || !d_A || !d_B || !d_C || !d_R || !d_Rm || !d_Y || !d_Z || !d_bits || !io) return RA_E_INVAL;
    if (!is_pow2(n) || !is_pow2(m) || !is_pow2(k)) return RA_E_INVAL;
    if (a_dtype != RA_I16 && a_dtype != RA_I32) return RA_E_INVAL;
    if (io->s < 1 || io->relu > 1 || io->round_mode > 1 || io->t < -1) return RA_E_INVAL;
    if (m > kGemmMaxInner || (uint64_t)n * k > kRangeMaxN || io->s > 16) return RA_E_NOT_IMPLEMENTED;
    if (c->phase != 0) return RA_E_STATE;
    const uint64_t N = (uint64_t)n * k;
    if (bits_words < N) return RA_E_BUFSIZE;
    const int ln = log2u(n), lm = log2u(m), lk = log2u(k), lN = ln + lk, relu = (int)io->relu;
    if ((lm && !io->mm_evals) || !io->rs_evals || (relu && lN && !io->zc_evals)) return RA_E_INVAL;
    ra_status st = drain(c);  // a synchronous call: earlier deferred outputs are completed first
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    const Fp2Layout L = fp2_layout(a_dtype == RA_I32, n, m, k);
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, L.bytes, &ws)) != RA_OK) return st;
    hipStream_t s = c->stream;
    auto tab = [&](size_t off, size_t len) {
        uint64_t *b = (uint64_t *)(ws + off);
        return F2Tab{b, b + len};
    };
    const uint64_t H = N > 1 ? N / 2 : 1;
    const F2Tab E1 = tab(L.o_e1, n), E2 = tab(L.o_e2, k), Ta = tab(L.o_a, m), Tb = tab(L.o_b, m);
    const F2Tab EQ = tab(L.o_eq, N), EQr = tab(L.o_eqr, H), EQz = tab(L.o_eqz, H), Bx = tab(L.o_bx, N);
    const F2Tab Dt = tab(L.o_d, H), St = tab(L.o_s, H), SIG = tab(L.o_sig, 64), ONE = tab(L.o_one, 1);
    uint64_t *scr = (uint64_t *)(ws + L.o_scr), *part = (uint64_t *)(ws + L.o_part);
    uint64_t *cpart = (uint64_t *)(ws + L.o_cpart), *cst = (uint64_t *)(ws + L.o_cst);
    uint64_t *tr = (uint64_t *)(ws + L.o_tr), *Gre = (uint64_t *)(ws + L.o_g), *Gim = Gre + 4096;
    const size_t pstride = (size_t)kF2MaxBlocks * 8;

    // the witness: the exact product, then t and P (given: fixed on the host)
    launch_gemm_mfma(d_A, a_dtype == RA_I32, d_B, d_C, n, m, k, ws + L.o_gemm, s, nullptr, nullptr, false, nullptr);
    int P = 0, lP = 0, t = io->t;
    WitParams hp{};
    if (t >= 0) {
        if ((st = plane_params((int)io->s, t, relu, &P, &lP)) != RA_OK) return st;
        hp.status = 0;
        hp.t = t;
        hp.P = P;
        hp.lP = lP;
        hp.s = (int)io->s;
        hp.relu = relu;
        hp.mode = (int)io->round_mode;
        hp.t_in = t;
    } else {
        launch_witness_params(d_C, N, (int)io->s, relu, (int)io->round_mode, -1, (int64_t *)(c->d_wit + kWitMinMax),
                              c->d_params, s);
        WitParams got;
        RA_HIP(hipMemcpyAsync(&got, c->d_params, sizeof(got), hipMemcpyDeviceToHost, s));
        RA_HIP(hipStreamSynchronize(s));
        if (got.status != 0) return got.status;
        t = got.t;
        P = got.P;
        lP = got.lP;
    }
    // the challenges, two words each
    const uint64_t cnt = (uint64_t)ln + lk + lm + 4 + 2 * lP + lN + (relu ? lN : 0);
    if ((st = ensure_chal(c, 2 * cnt)) != RA_OK) return st;
    const uint64_t *r1 = c->d_chal + c->cursor, *r2 = r1 + 2 * ln, *rho = r2 + 2 * lk, *lam = rho + 2 * lm;
    const uint64_t *tau = lam + 8, *sig = tau + 2 * lP, *rho2 = sig + 2 * (lP + lN);

    launch_f2_eq(r1, ln, E1, s);
    launch_f2_eq(r2, lk, E2, s);
    // R, Rm, Y, Z, the bit table (the F_p claims this pass also forms are not used)
    launch_witness_rescale(d_C, N, lk, E1.re, E2.re, d_R, d_Rm, d_Y, d_Z, d_bits, (uint64_t *)(c->d_wit + kWitClaims),
                           c->d_params, c->d_claims, nullptr, s, io->t >= 0 ? &hp : nullptr,
                           (uint32_t *)(c->d_wit + kWitFlags), nullptr);

    // matrix instance: a = the rows of A bound at r1, b = the columns of B at
    // r2 (two F_p bindings each), log m rounds
    launch_bind_rows(d_A, a_dtype, n, m, E1.re, scr, Ta.re, s);
    launch_bind_rows(d_A, a_dtype, n, m, E1.im, scr, Ta.im, s);
    launch_bind_cols(d_B, RA_I16, m, k, E2.re, Tb.re, s);
    launch_bind_cols(d_B, RA_I16, m, k, E2.im, Tb.im, s);
    uint64_t *ev_mm = tr + kF2TrFixed, *ev_rs = ev_mm + 6 * (size_t)lm, *ev_zc = ev_rs + 8 * (size_t)(lP + lN);
    uint64_t *p_mm = part, *p_rs = p_mm + (size_t)lm * pstride, *p_zc = p_rs + (size_t)lN * pstride;
    // each instance: one launch per round while its tables hold more than
    // 2^kF2TailLog entries, then the rest in one workgroup
    const int tm = std::min(lm, kF2TailLog), jm = lm - tm;
    for (int j = 0; j < jm; j++) {
        F2RoundArgs ra{};
        ra.kind = F2_MATMUL;
        ra.h = (uint64_t)m >> (j + 1);
        ra.src[0] = ra.dst[0] = Ta;
        ra.src[1] = ra.dst[1] = Tb;
        ra.rho = rho + 2 * j;
        ra.part = p_mm + (size_t)j * pstride;
        launch_f2_round(ra, s);
    }
    if (tm > 0) {
        F2TailArgs ta{};
        ta.kind = F2_MATMUL;
        ta.v = tm;
        ta.src[0] = ta.dst[0] = Ta;
        ta.src[1] = ta.dst[1] = Tb;
        ta.rho = rho + 2 * jm;
        ta.part = p_mm + (size_t)jm * pstride;
        launch_f2_tail(ta, s);
    }
    {
        F2FinishArgs fa{};
        fa.kind = F2_MATMUL;
        fa.v = lm;
        fa.part = p_mm;
        fa.ev = ev_mm;
        fa.t[0] = Ta;
        fa.t[1] = Tb;
        fa.fin = tr;
        launch_f2_finish(fa, s);
    }
    // the claims at (r1, r2)
    launch_f2_outer(E1, E2, lk, N, EQ, s);
    launch_f2_claims(EQ, d_R, d_Rm, d_Y, d_Z, N, cpart, s);
    launch_f2_sum8(cpart, f2_blocks(N), tr + 6, s);
    // plane rounds: the Gram matrix's two parts from EQ's two parts (the F_p
    // Gram pass with EQ as its row table and a one-entry column table), and
    // the plane-bound table Bx with the two parts of eq(sigma_p, .)
    launch_f2_eq(sig, lP, SIG, s);
    launch_f2_eq(sig, 0, ONE, s);
    const int pused = (int)io->s + (t + 2) * (relu ? 2 : 1);  // planes the witness writes
    const int gt = plane_gram_tiles(lP, pused), gb = plane_gram_blocks(N, lP);
    uint64_t *gp0 = (uint64_t *)(ws + L.o_gp0), *gp1 = (uint64_t *)(ws + L.o_gp1);
    launch_plane_gram(lP, d_bits, N, 0, EQ.re, ONE.re, sig, Bx.re, gp0, nullptr, s, SIG.re, pused);
    launch_f2_gram_sum(gp0, gb, gt, Gre, s);
    launch_plane_gram(lP, d_bits, N, 0, EQ.im, ONE.re, sig, Bx.im, gp1, nullptr, s, SIG.im, pused);
    launch_f2_gram_sum(gp1, gb, gt, Gim, s);
    {
        F2PlaneArgs pa{};
        pa.G_re = Gre;
        pa.G_im = Gim;
        pa.tau = tau;
        pa.sig = sig;
        pa.lam = lam;
        pa.claims = tr + 6;
        pa.s = (int)io->s;
        pa.t = t;
        pa.relu = relu;
        pa.P = P;
        pa.lP = lP;
        pa.ev = ev_rs;
        pa.cst = cst;
        pa.range_sum = tr + 14;
        launch_f2_planes(pa, s);
    }
    // rounds over x of the range instance (tables EQ, Bx), then the ReLU zero-check (EQ, D, S)
    const int tx = std::min(lN, kF2TailLog), jx = lN - tx;
    for (int j = 0; j < jx; j++) {
        F2RoundArgs ra{};
        ra.kind = F2_RANGE;
        ra.first = j == 0;
        ra.h = N >> (j + 1);
        ra.src[0] = j == 0 ? EQ : EQr;
        ra.dst[0] = EQr;
        ra.src[1] = ra.dst[1] = Bx;
        ra.rho = sig + 2 * (lP + j);
        ra.cst = cst;
        ra.part = p_rs + (size_t)j * pstride;
        launch_f2_round(ra, s);
    }
    if (tx > 0) {
        F2TailArgs ta{};
        ta.kind = F2_RANGE;
        ta.first = jx == 0;
        ta.v = tx;
        ta.src[0] = jx == 0 ? EQ : EQr;
        ta.dst[0] = EQr;
        ta.src[1] = ta.dst[1] = Bx;
        ta.rho = sig + 2 * (lP + jx);
        ta.cst = cst;
        ta.part = p_rs + (size_t)jx * pstride;
        launch_f2_tail(ta, s);
    }
    {
        F2FinishArgs fa{};
        fa.kind = F2_RANGE;
        fa.v = lN;
        fa.part = p_rs;
        fa.ev = ev_rs + 8 * (size_t)lP;
        fa.t[0] = EQr;
        fa.t[1] = Bx;
        fa.fin = tr + 16;
        launch_f2_finish(fa, s);
    }
    if (relu) {
        for (int j = 0; j < jx; j++) {
            F2RoundArgs ra{};
            ra.kind = F2_RELU;
            ra.first = j == 0;
            ra.h = N >> (j + 1);
            ra.src[0] = j == 0 ? EQ : EQz;
            ra.dst[0] = EQz;
            ra.src[1] = ra.dst[1] = Dt;
            ra.src[2] = ra.dst[2] = St;
            ra.R = d_R;
            ra.Y = d_Y;
            ra.rho = rho2 + 2 * j;
            ra.part = p_zc + (size_t)j * pstride;
            launch_f2_round(ra, s);
        }
        if (tx > 0) {
            F2TailArgs ta{};
            ta.kind = F2_RELU;
            ta.first = jx == 0;
            ta.v = tx;
            ta.src[0] = jx == 0 ? EQ : EQz;
            ta.dst[0] = EQz;
            ta.src[1] = ta.dst[1] = Dt;
            ta.src[2] = ta.dst[2] = St;
            ta.R = d_R;
            ta.Y = d_Y;
            ta.rho = rho2 + 2 * jx;
            ta.part = p_zc + (size_t)jx * pstride;
            launch_f2_tail(ta, s);
        }
        F2FinishArgs fa{};
        fa.kind = F2_RELU;
        fa.v = lN;
        fa.part = p_zc;
        fa.ev = ev_zc;
        fa.t[0] = EQz;
        fa.t[1] = Dt;
        fa.t[2] = St;
        fa.fin = tr + 18;
        fa.R = d_R;
        fa.Y = d_Y;
        launch_f2_finish(fa, s);
    }
    RA_HIP(hipGetLastError());
    // the transcript and the witness status into the context's pinned area
    // (nothing else is pending there: the call drained on entry)
    const size_t prm_words = (sizeof(WitParams) + 7) / 8;
    size_t off = 0;
    if ((st = stage_take(c, L.tr_words + prm_words, &off)) != RA_OK) return st;
    const uint64_t *h = c->h_stage + off;
    RA_HIP(hipMemcpyAsync(c->h_stage + off, tr, L.tr_words * 8, hipMemcpyDeviceToHost, s));
    RA_HIP(hipMemcpyAsync(c->h_stage + off + L.tr_words, c->d_params, sizeof(WitParams), hipMemcpyDeviceToHost, s));
    RA_HIP(hipStreamSynchronize(s));
    WitParams prm;
    std::memcpy(&prm, h + L.tr_words, sizeof(prm));
    c->stage_used = 0;
    if (prm.status != 0) return prm.status;  // a given t that does not hold R
    c->cursor += 2 * cnt;
    c->link_ok = false;
    auto pr = [&](size_t o) { return ra_fp2{h[o], h[o + 1]}; };
    io->t = t;
    io->P = (uint32_t)P;
    io->log_m = (uint32_t)lm;
    io->c0 = pr(0);
    io->a_star = pr(2);
    io->b_star = pr(4);
    io->r_claim = pr(6);
    io->rm_claim = pr(8);
    io->y_claim = pr(10);
    io->z_claim = pr(12);
    io->range_sum = pr(14);
    io->bits_claim = pr(16);
    io->r_at = relu ? pr(18) : ra_fp2{0, 0};
    io->y_at = relu ? pr(20) : ra_fp2{0, 0};
    io->rounds = (uint32_t)(lP + lN);
    io->relu_rounds = relu ? (uint32_t)lN : 0;
    const size_t omm = kF2TrFixed, ors = omm + 6 * (size_t)lm, ozc = ors + 8 * (size_t)(lP + lN);
    for (int i = 0; i < 3 * lm; i++) io->mm_evals[i] = pr(omm + 2 * i);
    for (int i = 0; i < 4 * (lP + lN); i++) io->rs_evals[i] = pr(ors + 2 * i);
    if (relu)
        for (int i = 0; i < 4 * lN; i++) io->zc_evals[i] = pr(ozc + 2 * i);
    return RA_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The non-interactive layer proof (fs.hip): the F_{p^2} protocol with every
// challenge drawn on the device from the context's Fiat-Shamir transcript.
// ---------------------------------------------------------------------------
extern "C" ra_status ra_prove_layer_fs(ra_ctx *c, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                                       uint32_t m, uint32_t k, int64_t *d_C, int32_t *d_R, uint16_t *d_Rm,
                                       int32_t *d_Y, int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words,
                                       const uint8_t *pub_digest, void *d_ws, size_t ws_bytes,
                                       ra_layer_proof_fp2 *io, uint8_t *root_out)
{
    if (!c || !d_A || !d_B || !d_C || !d_R || !d_Rm || !d_Y || !d_Z || !d_bits || !io || !pub_digest)
        return RA_E_INVAL;
    if (!is_pow2(n) || !is_pow2(m) || !is_pow2(k)) return RA_E_INVAL;
    if (a_dtype != RA_I16 && a_dtype != RA_I32) return RA_E_INVAL;
    if (io->s < 1 || io->relu > 1 || io->round_mode > 1 || io->t < -1) return RA_E_INVAL;
    if (m > kGemmMaxInner || (uint64_t)n * k > kRangeMaxN || io->s > 16) return RA_E_NOT_IMPLEMENTED;
    if (!c->d_fs || c->phase != 0) return RA_E_STATE;
    const uint64_t N = (uint64_t)n * k;
    if (bits_words < N) return RA_E_BUFSIZE;
    const int ln = log2u(n), lm = log2u(m), lk = log2u(k), lN = ln + lk, relu = (int)io->relu;
    if ((lm && !io->mm_evals) || !io->rs_evals || (relu && lN && !io->zc_evals)) return RA_E_INVAL;
    ra_status st = drain(c);
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    const Fp2Layout L = fp2_layout(a_dtype == RA_I32, n, m, k);
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, L.bytes, &ws)) != RA_OK) return st;
    hipStream_t s = c->stream;
    auto tab = [&](size_t off, size_t len) {
        uint64_t *b = (uint64_t *)(ws + off);
        return F2Tab{b, b + len};
    };
    const uint64_t H = N > 1 ? N / 2 : 1;
    const F2Tab E1 = tab(L.o_e1, n), E2 = tab(L.o_e2, k), Ta = tab(L.o_a, m), Tb = tab(L.o_b, m);
    const F2Tab EQ = tab(L.o_eq, N), EQr = tab(L.o_eqr, H), EQz = tab(L.o_eqz, H), Bx = tab(L.o_bx, N);
    const F2Tab Dt = tab(L.o_d, H), St = tab(L.o_s, H), SIG = tab(L.o_sig, 64), ONE = tab(L.o_one, 1);
    uint64_t *scr = (uint64_t *)(ws + L.o_scr), *part = (uint64_t *)(ws + L.o_part);
    uint64_t *cpart = (uint64_t *)(ws + L.o_cpart), *cst = (uint64_t *)(ws + L.o_cst);
    uint64_t *tr = (uint64_t *)(ws + L.o_tr), *Gre = (uint64_t *)(ws + L.o_g), *Gim = Gre + 4096;
    uint64_t *fsch = (uint64_t *)(ws + L.o_fsch);
    uint32_t *err = (uint32_t *)(ws + L.o_err);
    uint8_t *root = (uint8_t *)(ws + L.o_root);

    // the witness: the exact product, t and P, then R, Rm, Y, Z and the bit
    // table (the F_p claims that pass also forms are not used: its eq tables
    // are zero here)
    launch_gemm_mfma(d_A, a_dtype == RA_I32, d_B, d_C, n, m, k, ws + L.o_gemm, s, nullptr, nullptr, false, nullptr);
    int P = 0, lP = 0, t = io->t;
    WitParams hp{};
    if (t >= 0) {
        if ((st = plane_params((int)io->s, t, relu, &P, &lP)) != RA_OK) return st;
        hp.status = 0;
        hp.t = t;
        hp.P = P;
        hp.lP = lP;
        hp.s = (int)io->s;
        hp.relu = relu;
        hp.mode = (int)io->round_mode;
        hp.t_in = t;
    } else {
        launch_witness_params(d_C, N, (int)io->s, relu, (int)io->round_mode, -1, (int64_t *)(c->d_wit + kWitMinMax),
                              c->d_params, s);
        WitParams got;
        RA_HIP(hipMemcpyAsync(&got, c->d_params, sizeof(got), hipMemcpyDeviceToHost, s));
        RA_HIP(hipStreamSynchronize(s));
        if (got.status != 0) return got.status;
        t = got.t;
        P = got.P;
        lP = got.lP;
    }
    launch_fill0(E1.re, n, s);
    launch_fill0(E2.re, k, s);
    launch_fill0((uint64_t *)err, 1, s);
    launch_witness_rescale(d_C, N, lk, E1.re, E2.re, d_R, d_Rm, d_Y, d_Z, d_bits, (uint64_t *)(c->d_wit + kWitClaims),
                           c->d_params, c->d_claims, nullptr, s, io->t >= 0 ? &hp : nullptr,
                           (uint32_t *)(c->d_wit + kWitFlags), nullptr);
    // the witness bound into the transcript before any challenge: its Merkle
    // root with the layer header and the caller's public digest; r1, r2
    MerkleArgs ma{};
    ma.seg[0] = MerkleSeg{(const uint8_t *)d_R, 4 * N, 0};
    ma.seg[1] = MerkleSeg{(const uint8_t *)d_Rm, 2 * N, 0};
    ma.seg[2] = MerkleSeg{(const uint8_t *)d_Y, 4 * N, 0};
    ma.seg[3] = MerkleSeg{(const uint8_t *)d_Z, 4 * N, 0};
    ma.seg[4] = MerkleSeg{(const uint8_t *)d_bits, 8 * N, 0};
    launch_merkle_root(ma, (uint32_t *)(ws + L.o_dig0), (uint32_t *)(ws + L.o_dig1), root, s);
    FsHeader hd{};
    const uint32_t hw[8] = {n, m, k, io->s, (uint32_t)relu, io->round_mode, (uint32_t)t, (uint32_t)P};
    for (int i = 0; i < 8; i++)
        for (int j = 0; j < 4; j++) hd.bytes[4 * i + j] = (uint8_t)(hw[i] >> (8 * j));
    std::memcpy(hd.bytes + 32, pub_digest, 32);
    // the layer's challenges (pairs), in the protocol's order
    uint64_t *r1 = fsch, *r2 = r1 + 2 * ln, *rho = r2 + 2 * lk, *lam = rho + 2 * lm, *tau = lam + 8;
    uint64_t *sig = tau + 2 * lP, *rho2 = sig + 2 * (lP + lN);
    launch_fs_header(c->d_fs, hd, root, r1, ln + lk, err, s);
    launch_f2_eq(r1, ln, E1, s);
    launch_f2_eq(r2, lk, E2, s);

    // matrix instance: each round folds the previous round's variable, then
    // evaluates; its values are hashed into the next challenge
    launch_bind_rows(d_A, a_dtype, n, m, E1.re, scr, Ta.re, s);
    launch_bind_rows(d_A, a_dtype, n, m, E1.im, scr, Ta.im, s);
    launch_bind_cols(d_B, RA_I16, m, k, E2.re, Tb.re, s);
    launch_bind_cols(d_B, RA_I16, m, k, E2.im, Tb.im, s);
    uint64_t *ev_mm = tr + kF2TrFixed, *ev_rs = ev_mm + 6 * (size_t)lm, *ev_zc = ev_rs + 8 * (size_t)(lP + lN);
    for (int j = 0; j < lm; j++) {
        F2FsRoundArgs ra{};
        ra.kind = F2_MATMUL;
        ra.fold = j > 0;
        ra.h = (uint64_t)m >> (j + 1);
        ra.src[0] = ra.dst[0] = Ta;
        ra.src[1] = ra.dst[1] = Tb;
        ra.rho_prev = j > 0 ? rho + 2 * (j - 1) : nullptr;
        ra.part = part;
        launch_f2_round_fs(ra, s);
        launch_fs_round(part, f2_blocks(ra.h), 6, ev_mm + 6 * j, c->d_fs, rho + 2 * j, err, s);
    }
    {
        F2FsFinalArgs fa{};
        fa.kind = F2_MATMUL;
        fa.rounds = lm;
        fa.t[0] = Ta;
        fa.t[1] = Tb;
        fa.rho = lm ? rho + 2 * (lm - 1) : nullptr;
        fa.ev0 = ev_mm;
        fa.fin = tr;
        launch_f2_final_fs(fa, s);
    }
    // the claims at (r1, r2), then a*, b* and the claims absorbed; lambda,
    // mu, tau_p drawn
    launch_f2_outer(E1, E2, lk, N, EQ, s);
    launch_f2_claims(EQ, d_R, d_Rm, d_Y, d_Z, N, cpart, s);
    launch_f2_sum8(cpart, f2_blocks(N), tr + 6, s);
    launch_fs_absorb_draw(c->d_fs, tr + 2, 12, lam, 4 + lP, err, s);
    // plane rounds: the Gram matrix's two parts (their pass's plane-bound
    // output is not used: sigma_p does not exist yet), then the rounds, which
    // draw sigma_p as they go, then Bx with eq(sigma_p, .)
    launch_fill0(SIG.re, 64, s);
    launch_f2_eq(lam, 0, ONE, s);
    const int pused = (int)io->s + (t + 2) * (relu ? 2 : 1);  // planes the witness writes
    const int gt = plane_gram_tiles(lP, pused), gb = plane_gram_blocks(N, lP);
    uint64_t *gp0 = (uint64_t *)(ws + L.o_gp0), *gp1 = (uint64_t *)(ws + L.o_gp1);
    launch_plane_gram(lP, d_bits, N, 0, EQ.re, ONE.re, SIG.re, Bx.re, gp0, nullptr, s, SIG.re, pused);
    launch_f2_gram_sum(gp0, gb, gt, Gre, s);
    launch_plane_gram(lP, d_bits, N, 0, EQ.im, ONE.re, SIG.re, Bx.im, gp1, nullptr, s, SIG.re, pused);
    launch_f2_gram_sum(gp1, gb, gt, Gim, s);
    {
        F2PlaneArgs pa{};
        pa.G_re = Gre;
        pa.G_im = Gim;
        pa.tau = tau;
        pa.sig = sig;
        pa.lam = lam;
        pa.claims = tr + 6;
        pa.s = (int)io->s;
        pa.t = t;
        pa.relu = relu;
        pa.P = P;
        pa.lP = lP;
        pa.ev = ev_rs;
        pa.cst = cst;
        pa.range_sum = tr + 14;
        pa.fs = c->d_fs;
        pa.sig_out = sig;
        pa.err = err;
        launch_f2_planes(pa, s);
    }
    launch_f2_eq(sig, lP, SIG, s);
    launch_f2_bx(d_bits, N, SIG, P, Bx, s);
    // rounds over x of the range instance, then the ReLU zero-check
    for (int j = 0; j < lN; j++) {
        F2FsRoundArgs ra{};
        ra.kind = F2_RANGE;
        ra.fold = j > 0;
        ra.h = N >> (j + 1);
        ra.src[0] = j <= 1 ? EQ : EQr;
        ra.dst[0] = EQr;
        ra.src[1] = ra.dst[1] = Bx;
        ra.rho_prev = j > 0 ? sig + 2 * (lP + j - 1) : nullptr;
        ra.cst = cst;
        ra.part = part;
        launch_f2_round_fs(ra, s);
        launch_fs_round(part, f2_blocks(ra.h), 8, ev_rs + 8 * (size_t)(lP + j), c->d_fs, sig + 2 * (lP + j), err, s);
    }
    {
        F2FsFinalArgs fa{};
        fa.kind = F2_RANGE;
        fa.rounds = lN;
        fa.t[0] = lN >= 2 ? EQr : EQ;
        fa.t[1] = Bx;
        fa.rho = lN ? sig + 2 * (lP + lN - 1) : nullptr;
        fa.fin = tr + 16;
        launch_f2_final_fs(fa, s);
    }
    launch_fs_absorb_draw(c->d_fs, tr + 16, 2, nullptr, 0, err, s);
    if (relu) {
        for (int j = 0; j < lN; j++) {
            F2FsRoundArgs ra{};
            ra.kind = F2_RELU;
            ra.fold = j > 0;
            ra.ints = j <= 1;
            ra.h = N >> (j + 1);
            ra.src[0] = j <= 1 ? EQ : EQz;
            ra.dst[0] = EQz;
            ra.src[1] = ra.dst[1] = Dt;
            ra.src[2] = ra.dst[2] = St;
            ra.R = d_R;
            ra.Y = d_Y;
            ra.rho_prev = j > 0 ? rho2 + 2 * (j - 1) : nullptr;
            ra.part = part;
            launch_f2_round_fs(ra, s);
            launch_fs_round(part, f2_blocks(ra.h), 8, ev_zc + 8 * (size_t)j, c->d_fs, rho2 + 2 * j, err, s);
        }
        F2FsFinalArgs fa{};
        fa.kind = F2_RELU;
        fa.rounds = lN;
        fa.ints = lN <= 1;
        fa.t[0] = lN >= 2 ? EQz : EQ;
        fa.t[1] = Dt;
        fa.t[2] = St;
        fa.R = d_R;
        fa.Y = d_Y;
        fa.rho = lN ? rho2 + 2 * (lN - 1) : nullptr;
        fa.fin = tr + 18;
        launch_f2_final_fs(fa, s);
        launch_fs_absorb_draw(c->d_fs, tr + 18, 4, nullptr, 0, err, s);
    }
    RA_HIP(hipGetLastError());
    // the transcript, the witness status, the transcript status and the root
    // into the context's pinned area (nothing else is pending there)
    const size_t prm_words = (sizeof(WitParams) + 7) / 8;
    size_t off = 0;
    if ((st = stage_take(c, L.tr_words + prm_words + 5, &off)) != RA_OK) return st;
    uint64_t *h = c->h_stage + off;
    RA_HIP(hipMemcpyAsync(h, tr, L.tr_words * 8, hipMemcpyDeviceToHost, s));
    RA_HIP(hipMemcpyAsync(h + L.tr_words, c->d_params, sizeof(WitParams), hipMemcpyDeviceToHost, s));
    RA_HIP(hipMemcpyAsync(h + L.tr_words + prm_words, err, 4, hipMemcpyDeviceToHost, s));
    RA_HIP(hipMemcpyAsync(h + L.tr_words + prm_words + 1, root, 32, hipMemcpyDeviceToHost, s));
    RA_HIP(hipStreamSynchronize(s));
    WitParams prm;
    std::memcpy(&prm, h + L.tr_words, sizeof(prm));
    uint32_t e = 0;
    std::memcpy(&e, h + L.tr_words + prm_words, 4);
    c->stage_used = 0;
    if (prm.status != 0) return prm.status;  // a given t that does not hold R
    if (e) return RA_E_INVAL;                // a transcript message longer than the pending area
    if (root_out) std::memcpy(root_out, h + L.tr_words + prm_words + 1, 32);
    auto pr = [&](size_t o) { return ra_fp2{h[o], h[o + 1]}; };
    io->t = t;
    io->P = (uint32_t)P;
    io->log_m = (uint32_t)lm;
    io->c0 = pr(0);
    io->a_star = pr(2);
    io->b_star = pr(4);
    io->r_claim = pr(6);
    io->rm_claim = pr(8);
    io->y_claim = pr(10);
    io->z_claim = pr(12);
    io->range_sum = pr(14);
    io->bits_claim = pr(16);
    io->r_at = relu ? pr(18) : ra_fp2{0, 0};
    io->y_at = relu ? pr(20) : ra_fp2{0, 0};
    io->rounds = (uint32_t)(lP + lN);
    io->relu_rounds = relu ? (uint32_t)lN : 0;
    const size_t omm = kF2TrFixed, ors = omm + 6 * (size_t)lm, ozc = ors + 8 * (size_t)(lP + lN);
    for (int i = 0; i < 3 * lm; i++) io->mm_evals[i] = pr(omm + 2 * i);
    for (int i = 0; i < 4 * (lP + lN); i++) io->rs_evals[i] = pr(ors + 2 * i);
    if (relu)
        for (int i = 0; i < 4 * lN; i++) io->zc_evals[i] = pr(ozc + 2 * i);
    c->link_ok = false;
    return RA_OK;
}

// ---------------------------------------------------------------------------
// The gather link (link.hip): after a layer's three calls, the claim a* =
// A~(r1, rho) of its matrix sum-check is reduced to the previous output.
// ---------------------------------------------------------------------------
namespace {
struct LinkLayout {
    size_t o_W, o_T0, o_part, o_E, o_bad, bytes;
};

// n + m: the eq tables of the layer's (r1, rho); at most 2^31 + 2^15 words
LinkLayout link_layout(uint64_t nz, uint64_t eq_words)
{
    const int vz = log2u(nz);
    Carve cv;
    LinkLayout L{};
    L.o_W = cv.take<uint64_t>(nz);
    L.o_T0 = cv.take<uint64_t>(nz > 1 ? nz / 2 : 1);
    L.o_part = cv.take<uint64_t>((size_t)(vz > 0 ? vz : 1) * kLinkMaxBlocks * 3);
    L.o_E = cv.take<uint64_t>(eq_words);
    L.o_bad = cv.take<uint32_t>(1);
    L.bytes = cv.off;
    return L;
}
}  // namespace

extern "C" ra_status ra_link_gather(ra_ctx *c, const int32_t *d_Z, uint64_t z_entries, const int32_t *d_src,
                                    uint64_t a_entries, int32_t *d_A)
{
    if (!c || !d_Z || !d_src || !d_A) return RA_E_INVAL;
    if (!is_pow2(z_entries) || !a_entries) return RA_E_INVAL;
    launch_link_gather(d_Z, z_entries, d_src, a_entries, d_A, c->stream);
    RA_HIP(hipGetLastError());
    return RA_OK;
}

extern "C" ra_status ra_link_workspace_size(uint64_t z_entries, uint32_t n, uint32_t m, size_t *bytes)
{
    if (!bytes || !is_pow2(z_entries) || !is_pow2(n) || !is_pow2(m)) return RA_E_INVAL;
    if (z_entries > kRangeMaxN) return RA_E_NOT_IMPLEMENTED;
    *bytes = link_layout(z_entries, (uint64_t)n + m).bytes;
    return RA_OK;
}

extern "C" ra_status ra_link_prove(ra_ctx *c, const int32_t *d_Z, uint64_t z_entries, const int32_t *d_src,
                                   uint64_t a_entries, void *d_ws, size_t ws_bytes, ra_link_proof *out)
{
    if (!c || !d_Z || !d_src || !out) return RA_E_INVAL;
    if (!is_pow2(z_entries)) return RA_E_INVAL;
    if (z_entries > kRangeMaxN) return RA_E_NOT_IMPLEMENTED;
    if (c->phase != 0 || !c->link_ok) return RA_E_STATE;
    if (a_entries != (uint64_t)c->n * c->m) return RA_E_INVAL;
    const int vz = log2u(z_entries), ln = log2u(c->n), lm = log2u(c->m), lk = log2u(c->k);
    if (vz && !out->evals) return RA_E_INVAL;
    ra_status st = ensure_chal(c, (uint64_t)vz);
    if (st != RA_OK) return st;
    const LinkLayout L = link_layout(z_entries, (uint64_t)c->n + c->m);
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, L.bytes, &ws)) != RA_OK) return st;
    // the transcript goes to the pinned area: 3 vz round words, then claim,
    // Z~(y*), W~(y*) and the map's status
    const size_t words = 3 * (size_t)vz + 4;
    size_t off = 0;
    if ((st = stage_take(c, words, &off)) != RA_OK) return st;
    hipStream_t s = c->stream;
    // the eq tables of (r1, rho) go to the link's own workspace (the
    // context's eq area may still be read by the layer's deferred kernels)
    uint64_t *E1 = (uint64_t *)(ws + L.o_E), *E2 = E1 + c->n;
    const uint64_t *r1 = c->d_chal + c->r12_off, *rho = r1 + ln + lk;
    launch_eq_tables(r1, ln, E1, rho, lm, E2, s);
    LinkArgs la{};
    la.src = d_src;
    la.na = a_entries;
    la.lm = lm;
    la.E1 = E1;
    la.E2 = E2;
    la.Z = d_Z;
    la.vz = vz;
    la.W = (uint64_t *)(ws + L.o_W);
    la.T0 = (uint64_t *)(ws + L.o_T0);
    la.rho = c->d_chal + c->cursor;
    la.part = (uint64_t *)(ws + L.o_part);
    la.tr = c->d_stage + off;
    la.fin = la.tr + 3 * (size_t)vz;
    la.bad = (uint32_t *)(ws + L.o_bad);
    launch_link(la, s);
    c->cursor += (uint64_t)vz;
    c->link_ok = false;
    const ra_status r = finish(c, off, [out, vz](const uint64_t *h) {
        if (h[3 * vz + 3]) return (ra_status)RA_E_INVAL;  // a gather index outside [-1, z_entries)
        out->rounds = (uint32_t)vz;
        if (vz) std::memcpy(out->evals, h, 3 * (size_t)vz * 8);
        out->claim = h[3 * vz];
        out->z_at = h[3 * vz + 1];
        out->w_at = h[3 * vz + 2];
        return (ra_status)RA_OK;
    });
    if (r != RA_OK && !c->deferred) {  // a refused map consumes nothing
        c->cursor -= (uint64_t)vz;
        c->link_ok = true;
    }
    return r;
}

// ---------------------------------------------------------------------------
// Commitments (commit.hip)
// ---------------------------------------------------------------------------
namespace {
int commit_kind(ra_dtype d)
{
    switch (d) {
    case RA_I16: return 0;
    case RA_U16: return 1;
    case RA_I32: return 2;
    case RA_U64: return 3;
    default: return -1;
    }
}
}  // namespace

extern "C" ra_status ra_commit_generators(ra_ctx *c, const uint8_t *domain, uint64_t first, uint64_t count,
                                          void *d_gens)
{
    if (!c || !domain || !d_gens) return RA_E_INVAL;
    if (!count) return RA_OK;
    ra_status st = drain(c);
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    char *ws = nullptr;
    if ((st = call_ws(c, nullptr, 0, 256, &ws)) != RA_OK) return st;
    hipStream_t s = c->stream;
    launch_fill0((uint64_t *)ws, 1, s);
    launch_commit_generators(domain, first, count, (uint32_t *)d_gens, (uint32_t *)ws, s);
    RA_HIP(hipGetLastError());
    size_t off = 0;
    if ((st = stage_take(c, 1, &off)) != RA_OK) return st;
    RA_HIP(hipMemcpyAsync(c->h_stage + off, ws, 4, hipMemcpyDeviceToHost, s));
    RA_HIP(hipStreamSynchronize(s));
    uint32_t err = 0;
    std::memcpy(&err, c->h_stage + off, 4);
    c->stage_used = 0;
    return err ? RA_E_INVAL : RA_OK;  // a counter ran out (probability about 2^-256 per generator)
}

extern "C" ra_status ra_commit_workspace_size(ra_dtype dtype, size_t *bytes)
{
    const int kind = commit_kind(dtype);
    if (!bytes || kind < 0) return RA_E_INVAL;
    *bytes = msm_workspace_bytes(kind) + 256;
    return RA_OK;
}

extern "C" ra_status ra_commit(ra_ctx *c, const void *d_values, ra_dtype dtype, uint64_t n, const void *d_gens,
                               void *d_ws, size_t ws_bytes, uint8_t *out)
{
    const int kind = commit_kind(dtype);
    if (!c || (n && (!d_values || !d_gens)) || !out || kind < 0) return RA_E_INVAL;
    ra_status st = drain(c);
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    const size_t need = msm_workspace_bytes(kind) + 256;
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, need, &ws)) != RA_OK) return st;
    hipStream_t s = c->stream;
    uint8_t *dout = (uint8_t *)(ws + msm_workspace_bytes(kind));
    launch_commit(d_values, kind, n, (const uint32_t *)d_gens, ws, dout, s);
    RA_HIP(hipGetLastError());
    size_t off = 0;
    if ((st = stage_take(c, 8, &off)) != RA_OK) return st;
    RA_HIP(hipMemcpyAsync(c->h_stage + off, dout, 64, hipMemcpyDeviceToHost, s));
    RA_HIP(hipStreamSynchronize(s));
    std::memcpy(out, c->h_stage + off, 64);
    c->stage_used = 0;
    return RA_OK;
}

extern "C" ra_status ra_commit_batch_workspace_size(const int32_t *dtypes, uint32_t count, size_t *bytes)
{
    if (!dtypes || !bytes || count == 0) return RA_E_INVAL;
    if (count > (uint32_t)kCommitBatchMax) return RA_E_NOT_IMPLEMENTED;
    int kinds[kCommitBatchMax];
    for (uint32_t t = 0; t < count; t++)
        if ((kinds[t] = commit_kind((ra_dtype)dtypes[t])) < 0) return RA_E_INVAL;
    size_t offs[kCommitBatchMax];
    *bytes = msm_batch_offsets(kinds, (int)count, offs) + 64 * (size_t)count + 256;
    return RA_OK;
}

extern "C" ra_status ra_commit_batch(ra_ctx *c, const void *const *d_values, const int32_t *dtypes,
                                     const uint64_t *ns, uint32_t count, const void *d_gens, void *d_ws,
                                     size_t ws_bytes, uint8_t *out)
{
    if (!c || !d_values || !dtypes || !ns || !d_gens || !out || count == 0) return RA_E_INVAL;
    if (count > (uint32_t)kCommitBatchMax) return RA_E_NOT_IMPLEMENTED;
    int kinds[kCommitBatchMax];
    for (uint32_t t = 0; t < count; t++) {
        if ((kinds[t] = commit_kind((ra_dtype)dtypes[t])) < 0) return RA_E_INVAL;
        if (ns[t] && !d_values[t]) return RA_E_INVAL;
    }
    ra_status st = drain(c);
    if (st != RA_OK && c->deferred_err == RA_OK) c->deferred_err = st;
    size_t offs[kCommitBatchMax];
    const size_t tables = msm_batch_offsets(kinds, (int)count, offs);
    const size_t need = tables + 64 * (size_t)count + 256;
    char *ws = nullptr;
    if ((st = call_ws(c, d_ws, ws_bytes, need, &ws)) != RA_OK) return st;
    hipStream_t s = c->stream;
    uint8_t *dout = (uint8_t *)(ws + tables);
    launch_commit_batch(d_values, kinds, ns, (int)count, (const uint32_t *)d_gens, ws, dout, s);
    RA_HIP(hipGetLastError());
    size_t off = 0;
    if ((st = stage_take(c, 8 * count, &off)) != RA_OK) return st;
    RA_HIP(hipMemcpyAsync(c->h_stage + off, dout, 64 * (size_t)count, hipMemcpyDeviceToHost, s));
    RA_HIP(hipStreamSynchronize(s));
    std::memcpy(out, c->h_stage + off, 64 * (size_t)count);
    c->stage_used = 0;
    return RA_OK;
}
