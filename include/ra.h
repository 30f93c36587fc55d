/*
 * ra.h -- C ABI of the MI355X (gfx950) Range-Arithmetic prover.
 *
 * One layer of a fixed-point network is C = A B followed by the rounding
 * operator of Sec. II-A and an optional ReLU (Sec. III-B).  The prover
 * convinces a verifier of it with
 *   - a sum-check over the inner index of gamma(l) = a~(r1, l) b~(l, r2)
 *     (Sec. III-A-1, Eq. (4); Alg. 1 step 6),
 *   - one concatenated range sum-check over a bit table holding the shifted
 *     remainder (s bits), R + 2^(t+1) (t + 2 bits) and, with ReLU, Y = |R|
 *     (t + 2 bits) (Sec. III-A-2; Alg. 1 steps 11-12; Sec. III-B),
 *   - the ReLU square-equality zero-check of Eq. (6).
 * All arithmetic is in F_p with p = 2^61 - 1; field elements cross the ABI
 * as uint64_t in [0, p).
 *
 * Calling convention
 *   - Per layer: ra_sumcheck_matmul_prove, then ra_rescale_relu_witness,
 *     then ra_range_prove; layers in order.  Out of order -> RA_E_STATE.
 *   - Pointers named d_* are device pointers (caller-owned, on the device
 *     that was current when the context was created); h_* and the arrays
 *     inside the proof structs are host pointers (caller-owned).
 *   - All device work is ordered on the context's HIP stream.  By default
 *     every call synchronises before it returns, so its outputs are ready.
 *     In deferred mode (ra_ctx_set_deferred) the proving calls return once
 *     their work is enqueued and their host outputs are written at
 *     ra_ctx_sync.
 *   - A context is not thread-safe.  Contexts on one device may run
 *     concurrently on different streams.
 *   - Dimensions n, m, k are powers of two >= 1 (Sec. III-A-1 assumes
 *     powers of two; callers zero-pad, which leaves the proof sound and
 *     complete because zero rows/columns give C = 0).
 *   - Matrices are row-major.  A table of 2^v entries is a function on
 *     {0,1}^v whose first variable is the most significant index bit; a
 *     matrix entry (i, j) sits at index i * cols + j, so row bits come
 *     before column bits (worked example of Sec. III-A-1).
 *   - Every function returns RA_OK (0) or a negative ra_status; none throws
 *     or aborts.  After an error the context is left in its previous state
 *     unless the error is RA_E_HIP.
 */
#ifndef RA_H
#define RA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ra_status;
#define RA_OK 0
#define RA_E_INVAL (-1)             /* bad argument: null pointer, dimension not a power of two, ... */
#define RA_E_UNSUPPORTED_PRIME (-2) /* p != 2^61 - 1 */
#define RA_E_FIELD_TOO_SMALL (-3)   /* s + t + 3 > 61 bits of p (Theorem A.1, condition 1) */
#define RA_E_RANGE (-4)             /* R outside [-2^(t+1), 2^(t+1)) for a given t, or too many bit planes */
#define RA_E_SEED (-5)              /* challenge stream: seed 0, a given array exhausted, or a challenge >= p */
#define RA_E_HIP (-6)               /* a HIP runtime call failed */
#define RA_E_STATE (-7)             /* call out of the per-layer order */
#define RA_E_BUFSIZE (-8)           /* a caller buffer is too small */
#define RA_E_NOT_IMPLEMENTED (-9)   /* valid for the protocol, beyond this GPU path's limits (see below) */
#define RA_E_SCRATCH (-10)          /* the call needs more than the fixed scratch of ra_mle_bind_noalloc */
#define RA_E_NOMEM (-11)            /* device or host allocation failed */

typedef enum { RA_I16 = 1, RA_I32 = 2, RA_I64 = 3, RA_FIELD = 4, RA_U16 = 5, RA_U64 = 6 } ra_dtype;

/* Rounding operator.  RA_ROUND_NEAREST is R(x) = (x + 2^(s-1) - ((x + 2^(s-1))
 * mod 2^s)) / 2^s of Sec. II-A with the floor modulo; the shifted remainder
 * Rm = (x + 2^(s-1)) mod 2^s = E + 2^(s-1) lies in [0, 2^s).  RA_ROUND_FLOOR
 * is R(x) = floor(x / 2^s), Rm = x mod 2^s. */
typedef enum { RA_ROUND_NEAREST = 0, RA_ROUND_FLOOR = 1 } ra_round;

typedef struct ra_ctx ra_ctx;

/* Create a prover context.
 *   p           must be 2^61 - 1, else RA_E_UNSUPPORTED_PRIME.
 *   seed        state of the verifier's challenge stream (nonzero, else
 *               RA_E_SEED): xorshift64 with shifts 13, 7, 17 (Marsaglia,
 *               "Xorshift RNGs", 2003), each challenge the next 64-bit output
 *               reduced mod p.  The challenges are the verifier's coins of
 *               Alg. 1 step 4 and of every sum-check round of Sec. II-D,
 *               consumed in this order per layer: r1 (log n), r2 (log k),
 *               rho (log m), lambda1, lambda2, lambda3, mu, tau_p (log P),
 *               sigma (log P + log N), and with ReLU rho' (log N), where
 *               N = n k and P is the layer's bit-plane count.  The context
 *               draws them on the host and keeps them on the device, drawing
 *               more (after waiting for its stream) when a call needs them.
 *   hip_stream  hipStream_t to enqueue on (NULL = the null stream).
 *   out         receives the context.
 * Soundness note: the prover's witness tables (R, Rm, Y, Z, the bit table)
 * are a function of C alone, so they are fixed before r1, r2 are drawn; a
 * deployment that replaces the seeded coins by Fiat-Shamir must commit to
 * (absorb) those tables before deriving r1, r2 (Alg. 1 commits C' in step 7
 * before the checks that use the point), because the rounding link, the
 * output link, the recomposition and the zero-check test them only at (r1, r2). */
ra_status ra_ctx_create(uint64_t p, uint64_t seed, void *hip_stream, ra_ctx **out);
/* The same with the challenges given: h_challenges holds n_challenges field
 * elements in [0, p) (else RA_E_SEED), copied to the device once; a call that
 * needs more than remain returns RA_E_SEED. */
ra_status ra_ctx_create_stream(uint64_t p, const uint64_t *h_challenges, uint64_t n_challenges, void *hip_stream,
                               ra_ctx **out);
/* Device workspace (bytes) that covers every call of one layer with these
 * dimensions and at most P bit planes (int32 layer input and ReLU assumed),
 * for callers that pass their own workspace to the proving calls.  n, m, k,
 * P powers of two, else RA_E_INVAL. */
ra_status ra_workspace_size(uint32_t n, uint32_t m, uint32_t k, uint32_t P, size_t *bytes);
ra_status ra_ctx_destroy(ra_ctx *ctx);
/* Number of challenges consumed so far. */
ra_status ra_ctx_cursor(const ra_ctx *ctx, uint64_t *consumed);
const char *ra_status_str(ra_status st);

/* Deferred host outputs, for callers that pipeline many layers without
 * waiting on each call.
 *   ra_ctx_set_deferred(ctx, 1): from now on ra_sumcheck_matmul_prove and
 *     ra_range_prove return once their work is enqueued; ra_rescale_relu_witness does
 *     the same when the caller gives t (io->t >= 0: the plane count P is then
 *     known on the host and io->P is set at once), and otherwise waits for t
 *     and P as in synchronous mode.  A witness call that does not wait leaves
 *     the last sum of its claims to the range call that follows it (or to
 *     the next wait on the context); nothing else observes the difference.
 *     The kernels write transcripts straight into the context's pinned area,
 *     which grows (after writing out what is pending) when the calls kept
 *     pending outgrow it.  The caller keeps every proof struct, its
 *     evals arrays and the witness info alive and unread until ra_ctx_sync.
 *     Argument and state errors are still returned by the call itself; errors
 *     found on the device (a value outside the given range) are returned by
 *     ra_ctx_sync, after which the per-layer state of the context is not
 *     meaningful (create a new context to continue).
 *   ra_ctx_set_deferred(ctx, 0): completes what is pending and returns to
 *     synchronous calls (a device error found then is kept for ra_ctx_sync).
 *   ra_ctx_sync: waits for all enqueued work, writes every pending host
 *     output, and returns the first error met since the last ra_ctx_sync
 *     (RA_OK if none).  Harmless in synchronous mode. */
ra_status ra_ctx_set_deferred(ra_ctx *ctx, int on);
ra_status ra_ctx_sync(ra_ctx *ctx);

/* Kernel timing for benchmarks.  With profiling on, every group of kernel
 * launches (matrix product, bindings, witness passes, plane rounds, global
 * rounds, LDS tails, assembly) is bracketed by HIP events recorded on the
 * context's stream; the elapsed times are accumulated per group when each
 * call synchronises.  Turning profiling on or off clears the totals.
 *   ra_ctx_profile: group `index` (0-based; RA_E_INVAL past the last one)
 *   -> its name (static string), total milliseconds and launch count. */
ra_status ra_ctx_set_profiling(ra_ctx *ctx, int on);
ra_status ra_ctx_profile(const ra_ctx *ctx, uint32_t index, const char **name, double *total_ms,
                         uint64_t *launches);

/* Multilinear-extension binding of one side of a matrix (the chi-vector inner
 * product of Sec. II-C applied to every row or column):
 *   bind_rows = 1:  d_out[c] = sum_r eq(point, r) T[r, c],  point_len = log2(rows),
 *                   d_out has cols entries;
 *   bind_rows = 0:  d_out[r] = sum_c T[r, c] eq(point, c),  point_len = log2(cols),
 *                   d_out has rows entries;
 * with eq(z, y) = prod_i (z_i y_i + (1 - z_i)(1 - y_i)) (Eq. (1)).
 *   d_T     rows x cols, row-major, of dtype RA_I16 / RA_I32 / RA_I64
 *           (signed integers embedded in F_p) or RA_FIELD (uint64 in [0, p)).
 *   h_point point_len field elements in [0, p) (host).
 *   d_out   device, uint64 field elements.
 * Consumes no challenges.  RA_E_INVAL on a bad dimension, dtype or point. */
ra_status ra_mle_bind(ra_ctx *ctx, const void *d_T, ra_dtype dtype, uint32_t rows, uint32_t cols, int bind_rows,
                      const uint64_t *h_point, uint32_t point_len, uint64_t *d_out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * binding as ra_mle_bind, bit for bit, without a context.  It allocates
 * nothing and copies nothing: the point is passed to the kernels by value,
 * and the eq table (2^point_len words) and a row binding's chunk sums live in
 * a fixed device array of RA_NOALLOC_SCRATCH_BYTES per GPU, held by each GPU
 * the library runs on until the process ends.
 *   Arguments as for ra_mle_bind, plus hip_stream (hipStream_t; NULL = the
 *   null stream) on the current device.  The work is enqueued and the call
 *   returns without waiting: d_out is ready when the stream is.
 *   Every call on one GPU shares that GPU's array, so calls whose work
 *   overlaps on one GPU (other streams or threads) race; calls ordered on one
 *   stream do not.  Every word a call reads from the array it writes first.
 *   RA_E_SCRATCH when the eq table plus the row binding's chunk sums exceed
 *   the array (point_len <= 18 always fits); RA_E_INVAL as ra_mle_bind;
 *   RA_E_HIP if the array's device address cannot be found. */
#define RA_NOALLOC_SCRATCH_BYTES (4u << 20)
ra_status ra_mle_bind_noalloc(const void *d_T, ra_dtype dtype, uint32_t rows, uint32_t cols, int bind_rows,
                              const uint64_t *h_point, uint32_t point_len, uint64_t *d_out, void *hip_stream);

/* Transcript of the matrix-multiplication sum-check. */
typedef struct {
    uint32_t log_m;  /* out: number of rounds */
    uint64_t c0;     /* out: claimed sum  sum_l a~(r1, l) b~(l, r2) = C~(r1, r2) */
    uint64_t *evals; /* in: host buffer of 3 * log m words; out: g_j(0), g_j(1), g_j(2) per round */
    uint64_t a_star; /* out: a~(r1, rho) */
    uint64_t b_star; /* out: b~(rho, r2) */
} ra_matmul_proof;

/* Workspace of the three proving calls (d_ws, ws_bytes): NULL uses the
 * context's own device workspace, grown on demand; otherwise device memory
 * the caller owns, of at least ra_workspace_size bytes for the layer (else
 * RA_E_BUFSIZE), not used by anything else until the call's work has run on
 * the context's stream.  A call only uses it while its own kernels run. */

/* Alg. 1 steps 2 and 4-6 for one layer: computes the witness C = A B exactly
 * (int64), draws r1, r2, binds A's rows at r1 and B's columns at r2 (Eq. (4))
 * and runs the degree-2 sum-check over l in {0,1}^(log m), drawing rho.
 *   d_A     n x m, RA_I16 or RA_I32 (layer input; later layers use the
 *           previous int32 output).
 *   d_B     m x k int16 weights.
 *   d_C     out, n x k int64, the exact product.
 *   out     transcript; out->evals must hold 3 * log2(m) words.
 * The context keeps r1, r2 for the next two calls of this layer.
 * Limits of this GPU path (RA_E_NOT_IMPLEMENTED): m <= 32768 (the product
 * is formed exactly from 8-bit limbs with int32 partial sums) and
 * n k <= 2^31 (the layer's range call). */
ra_status ra_sumcheck_matmul_prove(ra_ctx *ctx, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                                   uint32_t m, uint32_t k, int64_t *d_C, void *d_ws, size_t ws_bytes,
                                   ra_matmul_proof *out);

/* Parameters and claims of the rescale / ReLU witness. */
typedef struct {
    uint32_t s;          /* in: fractional bits removed, >= 1 (this GPU path: <= 16) */
    uint32_t relu;       /* in: 1 = ReLU after the rescale */
    uint32_t round_mode; /* in: ra_round */
    int32_t t;           /* in: -1 = least t with R in [-2^(t+1), 2^(t+1)); >= 0 = given.  out: t used */
    uint32_t P;          /* out: bit planes, next power of two >= s + (t+2) (1 + relu) (this GPU path: <= 64) */
    uint64_t r_claim;    /* out: R~(r1, r2) */
    uint64_t rm_claim;   /* out: Rm~(r1, r2) */
    uint64_t y_claim;    /* out: Y~(r1, r2) */
    uint64_t z_claim;    /* out: Z~(r1, r2) */
} ra_witness_info;

/* Alg. 1 step 9 and the witness side of Sec. III-B: from C computes
 *   R  = rounded output (int32),  Rm = shifted remainder in [0, 2^s) (uint16),
 *   Y  = |R| (int32),  Z = ReLU(R) = (R + Y) / 2 with ReLU, else Z = R (int32,
 *        the layer's inference output),
 *   bits: one uint64 word per output x (index i * k + j); bit q of word x is
 *        plane q of x:  q in [0, s): bit q of Rm;  q in [s, s + t + 2):
 *        bit q - s of R + 2^(t+1);  with ReLU q in [s + t + 2, s + 2t + 4):
 *        bit q - s - t - 2 of Y;  higher planes are zero,
 * picks t (or checks the given one), and returns the claims at (r1, r2).
 *   bits_words  capacity of d_bits in words, at least n * k.
 * Errors: RA_E_RANGE if a given t does not hold R; RA_E_FIELD_TOO_SMALL if
 * s + t + 3 > 61 (Theorem A.1, condition 1); RA_E_INVAL if s = 0.
 * Limits of this GPU path (RA_E_NOT_IMPLEMENTED): s <= 16 (Rm is uint16),
 * t <= 29 (R, Y, Z are int32), P <= 64 (one bit word per output). */
ra_status ra_rescale_relu_witness(ra_ctx *ctx, const int64_t *d_C, uint32_t n, uint32_t k, int32_t *d_R,
                                  uint16_t *d_Rm, int32_t *d_Y, int32_t *d_Z, uint64_t *d_bits,
                                  uint64_t bits_words, void *d_ws, size_t ws_bytes, ra_witness_info *io);

/* Optional: announce the next ra_rescale_relu_witness call (same layer) before
 * its ra_sumcheck_matmul_prove, so that the witness of Alg. 1 step 9 and Sec.
 * III-B is computed inside the exact product, from each entry of C while it
 * is still in registers (C is still written).  Call it between layers (the
 * context expects a matrix call).  The arguments are those the witness call
 * will pass: s, relu, round_mode and a given t >= 0 (the plane count P
 * follows from them), and the output buffers with the capacity of d_bits.
 * The witness call then only sums its claims if its arguments are exactly
 * these (and bits_words covers n * k); any other witness call, or a product
 * the fusion does not take, runs the witness in full, so the results never
 * depend on the plan.  The plan is used by one layer.
 * Errors: RA_E_INVAL for a null buffer, t < 0 or parameters the witness call
 * would reject; RA_E_FIELD_TOO_SMALL / RA_E_NOT_IMPLEMENTED as that call
 * would return them for s and t; RA_E_STATE when called between a layer's
 * calls. */
ra_status ra_witness_plan(ra_ctx *ctx, uint32_t s, uint32_t relu, uint32_t round_mode, int32_t t, int32_t *d_R,
                          uint16_t *d_Rm, int32_t *d_Y, int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words);

/* Transcript of the range sum-check and the ReLU zero-check. */
typedef struct {
    uint32_t rounds;       /* out: log P + log N */
    uint64_t *evals;       /* in: host buffer of 4 * (log P + log N) words; out: g_j(0..3) */
    uint64_t range_sum;    /* out: claimed sum mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~) at (r1, r2) */
    uint64_t bits_claim;   /* out: b~(sigma), the bit table's extension at the final point */
    uint32_t relu_rounds;  /* out: log N with ReLU, else 0 */
    uint64_t *relu_evals;  /* in: host buffer of 4 * log N words (unused without ReLU); out */
    uint64_t r_at;         /* out: R~(rho') */
    uint64_t y_at;         /* out: Y~(rho') */
} ra_range_proof;

/* Alg. 1 steps 11-12 and Sec. III-B in sum-check form.  Over the table
 * b(q, x) (index q N + x, plane bits first) proves
 *   sum_{q,x} eq(tau, (q, x)) b (b - 1) + mu W(q) eq((r1, r2), x) b
 *     = mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~)(r1, r2)
 * with tau = (tau_p, r1, r2) and W(q) = lambda_group(q) 2^(bit of q), i.e.
 * booleanity of every bit and recomposition of every range-checked value;
 * then with ReLU the zero-check sum_x eq((r1, r2), x) (R(x)^2 - Y(x)^2) = 0
 * of Eq. (6).  Inputs are the buffers the witness call filled and its info;
 * as that call leaves them, the bit words are zero above the planes it writes
 * (s + t + 2, with ReLU s + 2t + 4), and the plane rounds rely on it (a
 * table with bits set there gives a transcript that does not verify).
 * Limit of this GPU path: N = n k <= 2^31 (the plane rounds' exact int32
 * sums), else RA_E_NOT_IMPLEMENTED. */
ra_status ra_range_prove(ra_ctx *ctx, const uint64_t *d_bits, const int32_t *d_R, const int32_t *d_Y, uint32_t n,
                         uint32_t k, const ra_witness_info *info, void *d_ws, size_t ws_bytes,
                         ra_range_proof *out);

/* ---- Gather links between layers -------------------------------------------
 * Sec. III-C chains layers through their outputs.  A convolution's input is a
 * gather of the previous output Z (im2col: each entry read by up to kh kw
 * patch positions, with zero padding; flattening: a permutation); the paper
 * says nothing about proving it.  With A[a] = Z[src[a]] (A[a] = 0 where
 * src[a] = -1), the claim a* = A~(r1, rho) that the layer's matrix sum-check
 * ends in equals sum_y Z[y] W[y], W[y] = sum over the a with src[a] = y of
 * eq((r1, rho), a) (a = row * m + col, row variables first).  A degree-2
 * sum-check (Sec. II-D) over the entries of Z reduces it to Z~(y*) W~(y*) at
 * the point y* of its challenges: Z~(y*) is a claim on the previous output,
 * and the verifier computes W~(y*) from the public map. */
typedef struct {
    uint32_t rounds; /* out: log2 z_entries */
    uint64_t *evals; /* in: host buffer of 3 log2 z_entries words; out: g_j(0), g_j(1), g_j(2) */
    uint64_t claim;  /* out: g_1(0) + g_1(1) = A~(r1, rho), the layer's a* */
    uint64_t z_at;   /* out: Z~(y*) */
    uint64_t w_at;   /* out: W~(y*) */
} ra_link_proof;

/* Prove the gather link of the layer whose three calls (F_p) have just been
 * made: d_Z is the previous layer's output (z_entries int32, a power of
 * two, at most 2^31, row-major), d_src the layer's gather map (a_entries =
 * n m int32 indices into d_Z, or -1), both device pointers owned by the
 * caller.  Call it after the layer's ra_range_prove and before the next
 * proving call (RA_E_STATE otherwise); it consumes log2 z_entries challenges.
 * Outputs as for the proving calls: complete on return, or at ra_ctx_sync in
 * deferred mode (out and out->evals must stay valid until then).  An index
 * outside [-1, z_entries) is not followed and makes the call's status
 * RA_E_INVAL (a synchronous call then consumes no challenges).  Workspace
 * as for the proving calls (ra_link_workspace_size bytes for the layer's n,
 * m, or NULL for the context's own). */
ra_status ra_link_prove(ra_ctx *ctx, const int32_t *d_Z, uint64_t z_entries, const int32_t *d_src,
                        uint64_t a_entries, void *d_ws, size_t ws_bytes, ra_link_proof *out);
ra_status ra_link_workspace_size(uint64_t z_entries, uint32_t n, uint32_t m, size_t *bytes);
/* The gathered input itself on the device: d_A[a] = d_Z[d_src[a]], 0 where
 * d_src[a] = -1 (a_entries int32 outputs, caller-owned).  Enqueued on the
 * context's stream, ordered with its proving calls, returns at once; an
 * index outside [-1, z_entries) is not followed (d_A[a] = 0) and
 * ra_link_prove refuses the map. */
ra_status ra_link_gather(ra_ctx *ctx, const int32_t *d_Z, uint64_t z_entries, const int32_t *d_src,
                         uint64_t a_entries, int32_t *d_A);

/* ---- Commitments to the tables: Pedersen vectors on secp256k1 --------------
 * Sec. II-C commits a vector a by g^a with public generators g of a group in
 * which discrete logarithms are hard; Sec. IV instantiates the group with
 * secp256k1 (or BLS12-381).  Here, additively, P = sum_i v_i G_i on
 * y^2 = x^3 + 7 over F_q, q = 2^256 - 2^32 - 977, for integer tables v.
 * Generators: G_i = (x, y) for the first counter c = 0, 1, ... with which
 * x = SHA-256("range-arithmetic generators v1" || domain || LE64(i) ||
 * LE32(c)) (big-endian, mod q) has x^3 + 7 a square; y is the even root.
 * A point is returned as 64 big-endian bytes, x then y (the identity as 64
 * zero bytes).  These commitments are computed and opened here; the
 * sum-checks of this library run over F_p, p = 2^61 - 1, which is not the
 * curve's scalar field, so the openings that would replace the opened tables
 * (Alg. 2, 3) are not built. */

/* Generators first .. first + count - 1 of `domain` (32 host bytes) into
 * d_gens (device, caller-owned): count x 64 bytes, each x then y as eight
 * little-endian uint32 limbs (the layout ra_commit reads).  Waits for its
 * work. */
ra_status ra_commit_generators(ra_ctx *ctx, const uint8_t *domain, uint64_t first, uint64_t count, void *d_gens);
/* Workspace of ra_commit for a value type (RA_I16, RA_U16, RA_I32, RA_U64). */
ra_status ra_commit_workspace_size(ra_dtype dtype, size_t *bytes);
/* P = sum_{i < n} v_i G_i: d_values n device values of dtype (RA_I16,
 * RA_U16, RA_I32 or RA_U64: the tables R, Y, Z, Rm, the bit words),
 * d_gens at least n generators (ra_commit_generators).  out: 64 host bytes.
 * Waits for its work. */
ra_status ra_commit(ra_ctx *ctx, const void *d_values, ra_dtype dtype, uint64_t n, const void *d_gens, void *d_ws,
                    size_t ws_bytes, uint8_t *out);
/* Commitments to several tables in one call, each as ra_commit (Sec. II-C,
 * the Pedersen vector commitment g^a): table t has d_values[t] (device,
 * caller-owned), dtypes[t] (RA_I16, RA_U16, RA_I32 or RA_U64) and ns[t]
 * values, every table committed with the generators d_gens from generator 0
 * (at least max ns[t] of them).  The tables' bucket passes run one after
 * another; their bucket sums, bit sums and final doubling chains each run in
 * one launch for all tables, so the short serial parts of the tables overlap.
 * out: 64 host bytes per table, table t at out + 64 t, the same bytes
 * ra_commit gives.  count in 1 .. 64 (RA_E_INVAL for 0, a null pointer or an
 * unknown dtype; RA_E_NOT_IMPLEMENTED above 64).  Workspace:
 * ra_commit_batch_workspace_size.  Waits for its work. */
ra_status ra_commit_batch_workspace_size(const int32_t *dtypes, uint32_t count, size_t *bytes);
ra_status ra_commit_batch(ra_ctx *ctx, const void *const *d_values, const int32_t *dtypes, const uint64_t *ns,
                          uint32_t count, const void *d_gens, void *d_ws, size_t ws_bytes, uint8_t *out);
/* Host opening check: *ok = 1 if commitment (64 bytes) is sum_i v_i G_i for
 * the host values and generators (layouts as above), else 0. */
ra_status ra_commit_open(const void *h_values, ra_dtype dtype, uint64_t n, const void *h_gens,
                         const uint8_t *commitment, int32_t *ok);

/* ---- The protocol with challenges in the extension field F_{p^2} ----------
 * Sec. II-F asks for a field of more than 128 bits.  Over p = 2^61 - 1 a
 * cheating prover passes a sum-check round with probability about d / p
 * (Sec. II-D); with the verifier's challenges drawn from F_{p^2} = F_p[i] /
 * (i^2 + 1) (p = 3 mod 4, so x^2 + 1 is irreducible) it is about d / p^2,
 * about 2^-120 per round.  The witness (C, R, Rm, Y, Z, the bit table) is the
 * same integer data; every challenge-dependent value is an element of F_{p^2}.
 * Challenge j is read from the context's F_p stream as two consecutive
 * words, stream[2j] + stream[2j + 1] i, in the order of the F_p protocol. */
typedef struct {
    uint64_t re, im; /* re + im i, both in [0, p) */
} ra_fp2;

typedef struct {
    uint32_t s, relu, round_mode; /* in, as ra_witness_info */
    int32_t t;                    /* in: -1 = least t holding R, >= 0 = given; out: t used */
    uint32_t P;                   /* out: bit planes */
    uint32_t log_m;               /* out: rounds of the matrix instance */
    ra_fp2 c0, a_star, b_star;    /* out: as ra_matmul_proof */
    ra_fp2 *mm_evals;             /* in: host buffer of 3 log m elements; out: g_j(0..2) */
    ra_fp2 r_claim, rm_claim, y_claim, z_claim; /* out: R~, Rm~, Y~, Z~ at (r1, r2) */
    uint32_t rounds;              /* out: log P + log N */
    ra_fp2 *rs_evals;             /* in: host buffer of 4 (6 + log N) elements; out: g_j(0..3) */
    ra_fp2 range_sum, bits_claim; /* out */
    uint32_t relu_rounds;         /* out: log N with ReLU, else 0 */
    ra_fp2 *zc_evals;             /* in: host buffer of 4 log N elements (ReLU); out */
    ra_fp2 r_at, y_at;            /* out: R~(rho'), Y~(rho') */
} ra_layer_proof_fp2;

/* One whole layer (the three calls of the F_p protocol) with challenges in
 * F_{p^2}: the exact product d_C, the witness d_R, d_Rm, d_Y, d_Z, d_bits
 * (as ra_rescale_relu_witness), the matrix sum-check, the claims, the range
 * sum-check and with ReLU the zero-check, every transcript element in
 * F_{p^2}.  Call it between layers (RA_E_STATE otherwise); it waits for its
 * work and consumes 2 (log n + log k + log m + 4 + 2 log P + log N (1 + relu))
 * words of the stream.  Workspace as for the proving calls
 * (ra_workspace_size_fp2).  Errors and limits as for the three F_p calls. */
ra_status ra_prove_layer_fp2(ra_ctx *ctx, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                             uint32_t m, uint32_t k, int64_t *d_C, int32_t *d_R, uint16_t *d_Rm, int32_t *d_Y,
                             int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words, void *d_ws, size_t ws_bytes,
                             ra_layer_proof_fp2 *io);
ra_status ra_workspace_size_fp2(uint32_t n, uint32_t m, uint32_t k, size_t *bytes);

/* Public data of one layer for the verifier (host pointers). */
typedef struct {
    uint32_t n, m, k;
    uint32_t s, relu, round_mode;
    ra_dtype a_dtype;  /* RA_I16 or RA_I32 */
    const void *A;     /* n x m */
    const int16_t *B;  /* m x k */
    const int32_t *Z;  /* n x k, the claimed layer output */
    uint32_t chained;  /* 1: A must equal the previous layer's Z (int32) */
    const int32_t *link_src; /* NULL, or the gather map of A (n m indices into the previous layer's Z,
                                -1 = zero): a* is then checked by the layer's link proof, A not opened */
} ra_layer_public;

/* Opened tables standing in for the paper's commitments (host pointers). */
typedef struct {
    const int32_t *R;
    const uint16_t *Rm;
    const int32_t *Y;
    const uint64_t *bits; /* n * k words, layout of ra_rescale_relu_witness */
} ra_layer_tables;

typedef struct {
    ra_matmul_proof mm;
    ra_witness_info wit;
    ra_range_proof rng;
    ra_link_proof link; /* read when the layer's link_src is set */
} ra_layer_transcript;

/* Host-only verifier (Sec. IV).  Replays the challenge stream of `seed` (as
 * ra_ctx_create draws it; seed 0 -> RA_E_SEED), checks every
 * sum-check chain (g_j(0) + g_j(1) against the previous round's value at its
 * challenge, by Lagrange interpolation), every final identity, the rounding
 * link C~ = 2^s R~ + Rm~ - 2^(s-1) (floor mode: no offset), the output link
 * 2 Z~ = R~ + Y~ (or Z~ = R~), the field guard s + t + 3 <= 61, and opens the
 * tables by evaluating their multilinear extensions.
 *   *verdict      0 accept, else the first failing check:
 *                 1 matmul chain, 2 matmul final, 3 a-star / b-star opening, 4 rounding
 *                 link, 5 range chain, 6 range final identity, 7 bit-table
 *                 opening, 8 R/Rm/Y openings, 9 ReLU chain or final identity,
 *                 10 ReLU openings, 11 output link or Z opening, 12 parameters,
 *                 13 malformed layer, 14 chaining, 15 gather link (its chain from a*,
 *                 the final product, Z~(y*) against the previous layer's Z,
 *                 W~(y*) against the map).  A layer with a link consumes
 *                 log2 (previous n k) more challenges after its own.
 *   *failed_layer index of the failing layer (0 when accepted). */
ra_status ra_verify(uint64_t p, uint64_t seed, uint32_t n_layers, const ra_layer_public *pub,
                    const ra_layer_tables *tables, const ra_layer_transcript *tr, int32_t *verdict,
                    uint32_t *failed_layer);
/* The same with the challenges given (as for ra_ctx_create_stream); a stream
 * too short for the layers gives RA_E_SEED. */
ra_status ra_verify_stream(uint64_t p, const uint64_t *h_challenges, uint64_t n_challenges, uint32_t n_layers,
                           const ra_layer_public *pub, const ra_layer_tables *tables,
                           const ra_layer_transcript *tr, int32_t *verdict, uint32_t *failed_layer);

/* The host verifier for layers proven over F_{p^2} (ra_prove_layer_fp2): the
 * checks of ra_verify with the same verdict numbers, every transcript element
 * a pair (re, im) in [0, p), the challenges read from the stream of `seed` in
 * pairs.  Gather links are proven over F_p only: a layer with link_src set
 * gives verdict 13. */
ra_status ra_verify_fp2(uint64_t p, uint64_t seed, uint32_t n_layers, const ra_layer_public *pub,
                        const ra_layer_tables *tables, const ra_layer_proof_fp2 *tr, int32_t *verdict,
                        uint32_t *failed_layer);

/* ---- The non-interactive protocol: Fiat-Shamir over F_{p^2} ---------------
 * The paper's protocol is interactive (the verifier's coins; Sec. II-D, Alg.
 * 1).  Here every challenge is a hash of what the prover has sent before it.
 * With H = SHA-256 (FIPS 180-4):
 *   S = H("range-arithmetic fs v1" || domain), domain 32 caller bytes;
 *   absorb(M) appends M to the bytes Q pending since the last draw;
 *   a draw sets S = H(S || LE32(|Q|) || Q), empties Q and returns
 *   (LE64(S[0..8]) mod p) + (LE64(S[8..16]) mod p) i;
 *   F_{p^2} elements are absorbed as LE64(re) || LE64(im), integers as LE32.
 * Per layer, in order: absorb LE32 n, m, k, s, relu, round_mode, t, P, the
 * caller's 32-byte public digest (what binds A and B) and the Merkle root of
 * the witness tables; draw r1 (log n), r2 (log k); per matrix round absorb
 * g_j(0..2), draw rho_j; absorb a*, b*, R~, Rm~, Y~, Z~; draw lambda1..3, mu,
 * tau_p (log P); per range round absorb g_j(0..3), draw sigma_j; absorb
 * b~(sigma); with ReLU per round absorb g_j(0..3), draw rho'_j, then absorb
 * r_at, y_at.  The pending bytes carry into the next layer.
 * Merkle root: the tables R (LE32), Rm (LE16), Y (LE32), Z (LE32) and the bit
 * words (LE64), each zero-padded to 1024-byte chunks and concatenated; leaf
 * H(0x00 || chunk); while more than one digest remains, groups of 4 (the
 * last zero-filled) give H(0x01 || 4 digests); root H(0x02 || LE64(leaves)
 * || top).  The witness is thus fixed before any challenge that tests it. */

/* A context whose challenges come from a Fiat-Shamir transcript started
 * from `domain` (32 host bytes), carried from layer to layer on the device.
 * Only ra_prove_layer_fs draws from it (the stream calls return RA_E_SEED). */
ra_status ra_ctx_create_fs(uint64_t p, const uint8_t *domain, void *hip_stream, ra_ctx **out);

/* One layer's non-interactive proof: arguments, outputs and workspace
 * (ra_workspace_size_fp2) as ra_prove_layer_fp2, every challenge drawn on the
 * device from the context's transcript in the order above.  pub_digest: the
 * caller's 32 bytes binding the public inputs (host).  root_out (optional,
 * 32 host bytes): the witness tables' Merkle root.  Waits for its work;
 * RA_E_STATE on a context without a transcript. */
ra_status ra_prove_layer_fs(ra_ctx *ctx, const void *d_A, ra_dtype a_dtype, const int16_t *d_B, uint32_t n,
                            uint32_t m, uint32_t k, int64_t *d_C, int32_t *d_R, uint16_t *d_Rm, int32_t *d_Y,
                            int32_t *d_Z, uint64_t *d_bits, uint64_t bits_words, const uint8_t *pub_digest,
                            void *d_ws, size_t ws_bytes, ra_layer_proof_fp2 *io, uint8_t *root_out);

/* Host verifier of non-interactive proofs: replays each layer's transcript
 * (pub_digests: n_layers x 32 bytes) to recover its challenges, then applies
 * the checks of ra_verify_fp2 (same verdict numbers; 13 also for a transcript
 * that cannot be replayed). */
ra_status ra_verify_fs(uint64_t p, const uint8_t *domain, uint32_t n_layers, const ra_layer_public *pub,
                       const ra_layer_tables *tables, const ra_layer_proof_fp2 *tr, const uint8_t *pub_digests,
                       int32_t *verdict, uint32_t *failed_layer);

#ifdef __cplusplus
}
#endif

#endif /* RA_H */
