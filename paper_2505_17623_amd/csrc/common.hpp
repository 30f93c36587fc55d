// common.hpp -- declarations shared by the HIP kernel files and the host
// driver of the Range-Arithmetic prover.
#pragma once
#include <hip/hip_runtime.h>

#include "sha256.hpp"
#include <stddef.h>
#include <stdint.h>

namespace ra {

constexpr int kThreads = 256;          // block size of streaming kernels
constexpr int kTailThreads = 256;      // block size of the LDS tail kernel
constexpr int kTailMaxLog = 10;
constexpr int kTailMax = 1 << kTailMaxLog;  // largest table the single-workgroup tail takes
constexpr int kMaxBlocks = 1024;       // blocks of a grid-stride round kernel
constexpr int kXSplitLog = 12;         // x rounds: variables in the low part of the suffix eq heaps
constexpr int kXTailLog = 8;           // x rounds: the last pass binds at most this many variables
constexpr int kXBlockMax = 10;         // x rounds: variables bound by one workgroup in LDS (sub-cube 2^B)
constexpr int kXFuseMax = 4;           // x rounds fused per thread in registers
constexpr int kMaxUnits = 2048;        // partial-sum producers per round (waves or threads)
constexpr int kPartWidth = 8;          // words per block and round in a partial-sum slot


constexpr int kMaxSlots = 96;          // per-call partial-sum slots (rounds)
constexpr int kMaxPlaneLog = 6;        // bit planes per output <= 64 (one word)
// outputs per range call: the plane rounds' int32 digit sums of a block (at
// most 2^23 outputs of |digit| <= 128 per block at this N) stay exact
constexpr uint64_t kRangeMaxN = 1ull << 31;

// Constant block of the concatenated range check (words), see sumcheck.hip.
constexpr int C_E = 0;      // e_j[p'] = eq(tau_{>j}, p'), j = 1..lP, sizes P/2, P/4, ..., 1
constexpr int C_W = 64;     // W_j, sizes P, P/2, ..., 2
constexpr int C_W2 = 192;   // 2 W_j[i + h] - W_j[i], sizes P/2, ..., 1
constexpr int C_K = 256;    // K_j, j = 1..lP
constexpr int C_TAU = 264;  // tau_p
constexpr int C_EP = 272;   // Ep, c (the range summand over x), Wp, mu
constexpr int C_WORDS = 280;

// Sum-check instance kinds (see sumcheck.hip).
enum Kind { KIND_MATMUL = 0 };

// Parameters of the rescale / ReLU witness, written on the device.
struct WitParams {
    int32_t status;  // 0 ok, else an RA_E_* code
    int32_t t, P, lP;
    int32_t s, relu, mode, t_in;
    int64_t cmin, cmax;
};

// Where the per-block partial sums of one round live and how to combine them.
enum SlotKind {
    SLOT_COPY = 0,  // the reduced words are the round's evaluations
    SLOT_X = 1      // range / ReLU x round: eight sums turned into g(0..3) (xrounds.hip)
};
struct Slot {
    int32_t nblk;      // blocks (or threads) that wrote partials
    int32_t width;     // words per block
    int32_t out;       // offset of the round's evaluations in the transcript buffer
    int32_t kind;      // SlotKind
    int32_t round;     // SLOT_X: the round j over x
    int32_t sum_out;   // >= 0: also write g(0) + g(1) (the instance's claimed sum) there
    int32_t out2;      // SLOT_X with ReLU: offset of the ReLU round's evaluations, else -1
};

// Set-up of the rounds over x (xsetup.hpp): r the EQ point, sigma_x and rho'
// (nullptr without ReLU), lN variables, L of them in the low part.
struct XSetupArgs {
    const uint64_t *r, *sigx, *rho2;
    int lN, L, nhs;  // nhs = 2^(lN - L) (1 if lN <= L)
    uint64_t *HS, *LS, *Kr, *Kz;
    uint64_t *WS;    // weights of the LDS pass over rounds wj .. wj + wB - 1 (wB = 0: none)
    int wj, wB;
};

// ---- launchers (witness.hip) ----
void launch_eq_table(const uint64_t *z, int v, uint64_t *out, hipStream_t st);
// a point of at most 32 variables passed by value (kernel argument)
struct EqPoint {
    uint64_t z[32];
    int v;
};
void launch_eq_table_val(const EqPoint &pt, uint64_t *out, hipStream_t st);
// both tables of a product's two sides in one launch
void launch_eq_tables(const uint64_t *z1, int v1, uint64_t *out1, const uint64_t *z2, int v2, uint64_t *out2,
                      hipStream_t st);
// ---- launchers (gemm.hip) ----
constexpr uint32_t kGemmMaxInner = 32768;  // exactness bound of the int32 limb accumulators
size_t gemm_workspace_bytes(int a_is_i32, uint32_t n, uint32_t m, uint32_t k);
struct TailArgs;
struct XJobs;
// ta, jobs (optional): the matrix instance's tail (launch_tail) as extra
// workgroups of the product launch
// The rescale / ReLU witness fused into the product's epilogue
// (ra_witness_plan): parameters, the eq tables of (r1, r2), the outputs, and
// per output tile four claim partials and a range flag (claims.hpp).
struct WitEpi {
    int s, t, relu;
    int64_t half;
    const uint64_t *E1, *E2;
    int32_t *R;
    uint16_t *Rm;
    int32_t *Y, *Z;
    uint64_t *bits;
    uint64_t *claim_part;
    uint32_t *flags;
};
// Output tiles of the product (one workgroup and one witness partial each).
uint32_t gemm_tiles(uint32_t n, uint32_t k);
// split_done: the limb planes are already in ws (launch_front); we
// (optional): the witness fused into the epilogue
void launch_gemm_mfma(const void *A, int a_is_i32, const int16_t *B, int64_t *C, uint32_t n, uint32_t m, uint32_t k,
                      void *ws, hipStream_t st, const TailArgs *ta = nullptr, const XJobs *jobs = nullptr,
                      bool split_done = false, const WitEpi *we = nullptr);
// The fused front of the matrix call (one launch): the product's limb split
// into ws, the row binding of A at r1 added into acc (2 m words: low 32 bits,
// high bits; zero on entry), the column binding of B at r2 into b, and the
// eq tables E1 (n words) and E2 (k words).  front_supported tells whether the
// shapes and alignments allow it.
bool front_supported(int a_is_i32, uint32_t n, uint32_t m, uint32_t k, const void *A, const void *B);
void launch_front(const void *A, int a_is_i32, const int16_t *B, uint32_t n, uint32_t m, uint32_t k,
                  const uint64_t *r1, int ln, const uint64_t *r2, int lk, uint64_t *acc, uint64_t *b, uint64_t *E1,
                  uint64_t *E2, void *ws, hipStream_t st);
// rows binding: out[c] = sum_r E[r] T[r, c]; needs scratch of bind_rows_chunks(rows, cols) * cols words
int bind_rows_chunks(uint32_t rows, uint32_t cols);
void launch_bind_rows(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E, uint64_t *scratch,
                      uint64_t *out, hipStream_t st);
// The second pass of a row binding (out = sum of the chunk rows of part).
struct ChunkSum {
    const uint64_t *part;
    int nch;
    uint32_t cols;
    uint64_t *out;
};
// first pass of a row binding only; the returned ChunkSum finishes it
ChunkSum launch_bind_rows_chunks(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E,
                                 uint64_t *scratch, uint64_t *out, hipStream_t st);
// cs (optional): also finish a row binding, in the same launch where possible
void launch_bind_cols(const void *T, int dtype, uint32_t rows, uint32_t cols, const uint64_t *E, uint64_t *out,
                      hipStream_t st, const ChunkSum *cs = nullptr);
int witness_blocks(uint64_t N);
void launch_witness_params(const int64_t *C, uint64_t N, int s, int relu, int mode, int t_in, int64_t *mm_part,
                           WitParams *params, hipStream_t st);
// mirror (optional): 12 words, the parameters (words 0-7) and the claims (8-11).
// known (optional): parameters computed on the host for a given t (status 0);
// then no params pass runs before, the range of R is checked here (flags:
// witness_blocks(N) words) and the parameters are written to params.
struct ClaimsJob;
// defer (optional): the last step is not launched but returned there, for a
// later launch to run (ClaimsJob).
void launch_witness_rescale(const int64_t *C, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2, int32_t *R,
                            uint16_t *Rm, int32_t *Y, int32_t *Z, uint64_t *bits, uint64_t *claim_part,
                            WitParams *params, uint64_t *claims_out, uint64_t *mirror, hipStream_t st,
                            const WitParams *known = nullptr, uint32_t *flags = nullptr, ClaimsJob *defer = nullptr);

// ---- launchers (sumcheck.hip) ----
int round_blocks(uint64_t h);
size_t tail_capacity(int ntab);  // largest 2^v table size the LDS tail holds
// Arguments of one sum-check instance's global-round launch and of its tail.
struct InstArgs {
    uint64_t *t0, *t1, *t2;
    const uint64_t *rho, *kp;
    uint64_t *part;
    uint64_t *acc;  // optional: t0's values as accumulated by launch_front (read, turned into t0, cleared)
};
// The last v rounds (rounds j0 .. j0 + v - 1 of the instance): round j's
// D + 1 evaluations go to tr[ev + (D + 1) j], with sum_out >= 0 and j0 == 0
// also g_0(0) + g_0(1) to tr[sum_out]; the tables' final values to fin*.
struct TailArgs {
    const uint64_t *t0, *t1, *t2;
    int v;
    const uint64_t *rho;
    uint64_t *tr;
    int ev, j0, sum_out;
    uint64_t *fin0, *fin1, *fin2;
    uint64_t *acc;  // optional (j0 == 0 only): t0's values as accumulated by launch_front, read and cleared
};
int fused_rounds_max(int kind);
// C fused rounds over tables of size S (C <= fused_rounds_max); partials of
// round r at part + r * stride
// acc (optional): t0's values accumulated by launch_front (read, cleared)
void launch_rounds(int kind, int C, uint64_t *t0, uint64_t *t1, uint64_t *t2, uint64_t S, const uint64_t *rho,
                   const uint64_t *kp, uint64_t *part, int stride, hipStream_t st, uint64_t *acc = nullptr);
struct XJobs;
// The tail workgroup, plus one workgroup per slot in jobs (SLOT_COPY slots of
// the global rounds before it).
void launch_tail(int kind, const TailArgs &a, const XJobs &jobs, hipStream_t st);
// The witness's last step (claims.hpp): the claims summed from nblk
// workgroup partials (4 words each), the status from their range flags when
// t was given (known: parameters hp), written to prm, out (4 words) and the
// staged transcript words `mirror` (12 words: parameters, claims).
struct ClaimsJob {
    const uint64_t *part;
    int nblk;  // 0: no job
    WitParams *prm;
    uint64_t *out, *mirror;
    WitParams hp;
    int known;
    const uint32_t *flags;
};
void launch_claims_final(const ClaimsJob &j, hipStream_t st);
// Constant block of the plane rounds (rsetup.hpp): lambda/mu/tau_p/sigma_p at
// chal, the witness parameters and claims; writes cst (C_WORDS) and the
// claimed sum of the range instance.  cj (nblk > 0): the witness's deferred
// last step, run first by the same workgroup.
struct RangeConsts {
    const uint64_t *chal;
    const WitParams *prm;
    const uint64_t *claims;
    int lP;
    uint64_t *cst, *range_sum;
    ClaimsJob cj;
};
void init_kernel_attributes();
// Constants of SLOT_X rounds: kp = (Ep, c) of the range summand, r the EQ
// point, Kr / Kz the prefix products of the range and ReLU instances.
struct XConst {
    const uint64_t *kp, *r, *Kr, *Kz;
};
// Plane rounds of the range check, evaluated by extra workgroups of the
// first x-round launch (plane_round.hpp): G, sigma_p, the constant block,
// transcript words 0 .. 4 lP.  lP = 0: none.
struct PlaneArgs {
    const uint64_t *G, *sigma, *cst;
    uint64_t *tr;
    int lP;
};


// ---- launchers (xrounds.hip) ----
struct XArgs {
    uint64_t *bx, *d, *s;          // Bx in place; D, S (written by the first launch)
    const int32_t *R, *Y;          // integer R, Y (first launch)
    const uint64_t *HS, *LS;       // suffix eq heaps
    const uint64_t *r;             // EQ point (lN words)
    const uint64_t *rho_a, *rho_z; // binding challenges of the launch's first round
    uint64_t *part;
    int lN, L, j;                  // variables, low-part size, first round
};
// Work for extra workgroups of an x-round launch: assemble nslot slots whose
// partials lie at part + q * stride (q < nslot), then evaluate plane rounds
// 1 .. nplane (plane_round.hpp).
constexpr int kXJobsMax = 12;
struct XJobs {
    int nslot, nplane;
    const uint64_t *part;
    int stride;
    uint64_t *tr;
    XConst xc;
    PlaneArgs pa;
    Slot s[kXJobsMax];
};
int xround_units(uint64_t sub, bool relu);  // partial-sum producers of a register pass
// Range-call work that rides in the first register pass's launch, after its
// jobs: nred workgroups sum the Gram pass's partial tiles (gpart, nblk
// blocks, `tiles` 16 x 16 tiles) into gsum, one writes the constant block (rc), and
// with a deferred witness step (rc.cj.nblk > 0) one more sums its claims.
struct RangeRiders {
    const uint64_t *gpart;
    int nblk, tiles, nred;
    uint64_t *gsum;
    RangeConsts rc;
};
int range_riders(const RangeRiders &r);  // workgroups the riders take
// C rounds per thread in registers over a table of S entries (sub-cube i:
// entries i + t S / 2^C).
void launch_xrounds(int C, bool first, bool relu, const XArgs &a, uint64_t S, int stride, const XJobs &jobs,
                    hipStream_t st, const RangeRiders *riders = nullptr);
// B rounds per workgroup in LDS over a table of 2^lS entries: sub-cube k (one
// workgroup) holds entries k + t 2^(lS - B).  With lS == B it is the last
// pass: its rounds' evaluations go to tr and the bound values to fin_*.
struct XBlockArgs {
    uint64_t *bx, *d, *s;           // tables; the bound values are written to index k
    const int32_t *R, *Y;           // integer R, Y (first pass)
    const uint64_t *HS, *LS, *r;    // suffix eq heaps, EQ point
    const uint64_t *W;              // heap of the weights inside a sub-cube (table s at 2^s, s < B)
    const uint64_t *rho_a, *rho_z;  // binding challenges of the pass's first round
    uint64_t *part;                 // pass: round c's partials at part + c * stride + 8 k
    int stride;
    int lN, L, j, B, lS;
    uint64_t *tr;                   // last pass: round c at tr + out0 + 4 c (ReLU: out2 + 4 c)
    int out0, out2;
    uint64_t *fin_b, *fin_r, *fin_y;
    XConst xc;
};
void launch_xblock(bool relu, bool first, const XBlockArgs &a, const XJobs &jobs, hipStream_t st);

// ---- the protocol over F_{p^2} (fp2.hip) ----
// An F_{p^2} table as two F_p arrays (real and imaginary parts).
struct F2Tab {
    uint64_t *re, *im;
};
enum { F2_MATMUL = 0, F2_RANGE = 1, F2_RELU = 2 };
constexpr int kF2MaxBlocks = 512;  // blocks of a round launch (partials per round)
// blocks of a pass over h pairs (256 threads each, grid-stride beyond kF2MaxBlocks)
__host__ __device__ inline int f2_blocks(uint64_t h)
{
    const uint64_t b = (h + 255) / 256;
    return (int)(b < (uint64_t)kF2MaxBlocks ? (b ? b : 1) : kF2MaxBlocks);
}
// one round over tables of 2h entries: src -> dst (equal but for the first
// round of the range / ReLU instances); rho and cst point at pairs (re, im)
struct F2RoundArgs {
    int kind, first;
    uint64_t h;
    F2Tab src[3], dst[3];
    const int32_t *R, *Y;  // ReLU first round: D = R - Y, S = R + Y
    const uint64_t *rho;
    const uint64_t *cst;   // range: c_eq, c_w
    uint64_t *part;        // f2_blocks(h) x 8 words
};
// the last v rounds (v <= kF2TailLog) of an instance, from its round j0 on,
// in one workgroup: src -> dst as in F2RoundArgs (first: j0 == 0); rho: the
// challenges of rounds j0 .. j0 + v - 1; part: round j0's partial slots
constexpr int kF2TailLog = 10;
struct F2TailArgs {
    int kind, first, v;
    F2Tab src[3], dst[3];
    const int32_t *R, *Y;
    const uint64_t *rho;
    const uint64_t *cst;
    uint64_t *part;
};
void launch_f2_tail(const F2TailArgs &a, hipStream_t st);
// the evaluations of an instance's v rounds (partials of round j at part +
// j kF2MaxBlocks 8) and its final words
struct F2FinishArgs {
    int kind, v;
    const uint64_t *part;
    uint64_t *ev;
    F2Tab t[3];
    uint64_t *fin;
    const int32_t *R, *Y;  // ReLU with no rounds (one output): D, S from R, Y
};
struct F2PlaneArgs {
    const uint64_t *G_re, *G_im;      // 64 x 64
    const uint64_t *tau, *sig, *lam;  // pairs: tau_p, sigma_p, (lambda1, lambda2, lambda3, mu)
    const uint64_t *claims;           // R~, Rm~, Y~, Z~ (pairs)
    int s, t, relu, P, lP;
    uint64_t *ev;                     // lP rounds x 8 words
    uint64_t *cst;                    // out: c_eq, c_w
    uint64_t *range_sum;              // out: the claimed sum
    // Fiat-Shamir (fs != nullptr): sigma_p is drawn round by round from the
    // transcript (after each round's values) into sig_out instead of read
    sha::Transcript *fs = nullptr;
    uint64_t *sig_out = nullptr;
    uint32_t *err = nullptr;
};
void launch_f2_eq(const uint64_t *z, int v, F2Tab out, hipStream_t st);
void launch_f2_outer(F2Tab E1, F2Tab E2, int lk, uint64_t N, F2Tab out, hipStream_t st);
void launch_f2_claims(F2Tab EQ, const int32_t *R, const uint16_t *Rm, const int32_t *Y, const int32_t *Z, uint64_t N,
                      uint64_t *part, hipStream_t st);
void launch_f2_sum8(const uint64_t *part, int nb, uint64_t *out, hipStream_t st);
void launch_f2_round(const F2RoundArgs &a, hipStream_t st);
void launch_f2_finish(const F2FinishArgs &a, hipStream_t st);
void launch_f2_planes(const F2PlaneArgs &a, hipStream_t st);
void launch_f2_gram_sum(const uint64_t *gpart, int nblk, int TP, uint64_t *G, hipStream_t st);

// ---- the non-interactive layer proof (fs.hip) ----
struct MerkleSeg {
    const uint8_t *p;     // 16-byte aligned
    uint64_t bytes;
    uint64_t first_leaf;  // set by launch_merkle_root
};
struct MerkleArgs {
    MerkleSeg seg[5];
    uint64_t leaves;
};
uint64_t merkle_leaves(const MerkleArgs &a);
// dig0, dig1: merkle_leaves() x 8 words each; root: 32 bytes
void launch_merkle_root(MerkleArgs a, uint32_t *dig0, uint32_t *dig1, uint8_t *root, hipStream_t st);
struct FsHeader {
    uint8_t bytes[64];  // LE32 n, m, k, s, relu, round_mode, t, P, then the 32-byte public digest
};
void launch_fs_header(sha::Transcript *fs, const FsHeader &h, const uint8_t *root, uint64_t *out, int ndraw,
                      uint32_t *err, hipStream_t st);
void launch_fs_absorb_draw(sha::Transcript *fs, const uint64_t *w, int nw, uint64_t *out, int ndraw, uint32_t *err,
                           hipStream_t st);
void launch_fs_round(const uint64_t *part, int nb, int nw, uint64_t *ev, sha::Transcript *fs, uint64_t *out,
                     uint32_t *err, hipStream_t st);
// A round whose pass first binds the previous round's variable (fold, tables
// of 4h entries at src to 2h at dst) and then evaluates on h pairs.
struct F2FsRoundArgs {
    int kind, fold, ints;      // ints: the ReLU tables D, S are read from R, Y
    uint64_t h;
    F2Tab src[3], dst[3];
    const int32_t *R, *Y;
    const uint64_t *rho_prev;  // pair
    const uint64_t *cst;       // range: c_eq, c_w
    uint64_t *part;            // f2_blocks(h) x 8 words
};
void launch_f2_round_fs(const F2FsRoundArgs &a, hipStream_t st);
struct F2FsFinalArgs {
    int kind, rounds, ints;
    F2Tab t[3];
    const int32_t *R, *Y;
    const uint64_t *rho;  // the last challenge (rounds > 0)
    const uint64_t *ev0;  // the first round's values (matrix c0)
    uint64_t *fin;
};
void launch_f2_final_fs(const F2FsFinalArgs &a, hipStream_t st);
void launch_f2_bx(const uint64_t *bits, uint64_t N, F2Tab SIG, int P, F2Tab Bx, hipStream_t st);
void launch_fill0(uint64_t *p, uint64_t n, hipStream_t st);

// ---- the gather link between layers (link.hip) ----
constexpr int kLinkMaxBlocks = 512;  // blocks of a round launch (partials per round)
constexpr int kLinkTailLog = 11;     // the last rounds, over at most 2^11 entries, run in one workgroup
__host__ __device__ inline int link_blocks(uint64_t h)
{
    const uint64_t b = (h + kThreads - 1) / kThreads;
    return (int)(b < (uint64_t)kLinkMaxBlocks ? (b ? b : 1) : kLinkMaxBlocks);
}
struct LinkArgs {
    const int32_t *src;        // na gather indices into Z (-1: zero)
    uint64_t na;
    int lm;                    // log2 of the next layer's inner dimension m (a = row * m + col)
    const uint64_t *E1, *E2;   // eq tables of r1 (rows) and rho (columns)
    const int32_t *Z;          // the previous output, 2^vz entries
    int vz;
    uint64_t *W, *T0;          // 2^vz and 2^(vz-1) words
    const uint64_t *rho;       // vz round challenges
    uint64_t *part;            // vz x kLinkMaxBlocks x 3 words
    uint64_t *tr;              // out: 3 vz words
    uint64_t *fin;             // out: claim, Z~(y*), W~(y*), the map's status (nonzero: an index outside)
    uint32_t *bad;             // out: nonzero if a gather index is outside [-1, 2^vz)
};
void launch_link(const LinkArgs &a, hipStream_t st);
void launch_link_gather(const int32_t *Z, uint64_t nz, const int32_t *src, uint64_t na, int32_t *A, hipStream_t st);

// ---- launchers (planes.hip) ----
// The Gram pass works on 16 x 16 tiles of G on and above the diagonal: 3 for
// up to 32 planes, 6 when P = 64 but only the first 48 planes can hold set
// bits (pused, the planes the witness writes: s + t + 2, with ReLU
// s + 2t + 4; the bit words are zero above them), 10 for 64; each block of
// the pass writes kGramTileWords words per tile, and the reduction takes 16
// entries per workgroup.
constexpr int kGramTileWords = 256;
int plane_gram_tiles(int lP, int pused = 64);  // tiles of the Gram matrix (3, 6 or 10)
int plane_gram_blocks(uint64_t N, int lP);    // blocks of the Gram pass (each writes tiles * kGramTileWords words)
inline int gram_reduce_groups(int tiles) { return tiles * kGramTileWords / 16; }
// threads of the Gram pass that can run the set-up of the rounds over x
int plane_gram_set_up_threads(uint64_t N, int lP);
// Bx per x and the blocks' partial Gram tiles (plane_gram_blocks x tiles x
// kGramTileWords words); sig: sigma_p (lP words).  With xs (x_setup_count(*xs) at most
// plane_gram_set_up_threads), the pass also runs the set-up of the rounds
// over x, which depends on challenges only.
// eqs (optional): the P values eq(sigma_p, q) given instead of computed from sig.
void launch_plane_gram(int lP, const uint64_t *bits, uint64_t N, int lk, const uint64_t *E1, const uint64_t *E2,
                       const uint64_t *sig, uint64_t *Bx, uint64_t *gpart, const XSetupArgs *xs, hipStream_t st,
                       const uint64_t *eqs = nullptr, int pused = 64);
// the Gram matrix G (gsum: 64 x 64 words, both triangles) from the partial
// tiles; further workgroups run the set-up of the range check (rc, xs)
void launch_gram_reduce(int lP, uint64_t N, const uint64_t *gpart, uint64_t *gsum, const RangeConsts &rc,
                        const XSetupArgs &xs, hipStream_t st, int pused = 64);

}  // namespace ra
