/*
 * ra_oracle_fp2.c -- the layer protocol of ra_oracle.c with the verifier's
 * challenges drawn from the quadratic extension F_{p^2} = F_p[i] / (i^2 + 1).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; it shares no code with the GPU path.
 *
 * Why: the paper asks for a field of more than 128 bits (Sec. II-F; Sec. IV,
 * security parameters).  A sum-check round over a field F lets a cheating
 * prover pass with probability at most d / |F| (Schwartz-Zippel, Sec. II-D),
 * so over p = 2^61 - 1 each round gives about 2^-59 and over F_{p^2} about
 * 2^-120.  The witness (C, R, Rm, Y, Z, the bit table) consists of integers
 * and is the same as over F_p; only the challenges and everything computed
 * from them (eq tables, bound tables, round polynomials, claims, final
 * values) live in F_{p^2}.
 *
 * F_{p^2}: p = 2^61 - 1 is 3 mod 4, so -1 is not a square mod p and
 * x^2 + 1 is irreducible; an element is a + b i with a, b in F_p and
 * (a + b i)(c + d i) = (ac - bd) + (ad + bc) i.
 *
 * Challenges: the stream of field elements of F_p (the seeded xorshift64
 * stream reduced mod p) is read in pairs; challenge j is
 * chal[2j] + chal[2j + 1] i.  They are consumed in the order of the F_p
 * protocol: r1 (log n), r2 (log k), rho (log m), lambda1..3, mu, tau_p
 * (log P), sigma (log P + log N), and with ReLU rho' (log N).
 *
 * Style: as ra_oracle.c -- every base operation is a 128-bit product or sum
 * followed by "% p", every multilinear extension the Lagrange-basis sum of
 * Eq. (1), every sum-check the textbook round loop of Sec. II-D over fully
 * materialised tables.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "ra_oracle_fs.h"

typedef unsigned __int128 u128;

#define P2_P ((uint64_t)0x1FFFFFFFFFFFFFFFULL) /* 2^61 - 1 */

enum { P2_OK = 0, P2_E_INVAL = -1, P2_E_CHALLENGES = -5, P2_E_NOMEM = -10 };

/* the witness and the bit table, from ra_oracle.c (field independent) */
int orc_layer_witness(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu,
                      int mode, int t_in, int64_t *C, int64_t *R, int64_t *Rm, int64_t *Y, int64_t *Z, int *t_out,
                      int *P_out, int *lP_out);
void orc_fill_planes(uint8_t *bits, int64_t N, int P, int s, int t, int relu, const int64_t *R, const int64_t *Rm,
                     const int64_t *Y);

/* ------------------------------------------------------------------------ */
/* F_p and F_{p^2}.                                                          */
/* ------------------------------------------------------------------------ */
static uint64_t padd(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a + b) % P2_P); }
static uint64_t psub(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a + P2_P - b) % P2_P); }
static uint64_t pmul(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a * b) % P2_P); }
static uint64_t pint(int64_t z)
{
    int64_t r = z % (int64_t)P2_P;
    if (r < 0) r += (int64_t)P2_P;
    return (uint64_t)r;
}
static uint64_t ppow(uint64_t b, uint64_t e)
{
    uint64_t r = 1;
    while (e) {
        if (e & 1) r = pmul(r, b);
        b = pmul(b, b);
        e >>= 1;
    }
    return r;
}

typedef struct { uint64_t re, im; } f2; /* re + im i */

static f2 f2of(uint64_t a) { f2 r = {a, 0}; return r; }
static f2 f2int(int64_t z) { return f2of(pint(z)); }
static f2 f2add(f2 a, f2 b) { f2 r = {padd(a.re, b.re), padd(a.im, b.im)}; return r; }
static f2 f2sub(f2 a, f2 b) { f2 r = {psub(a.re, b.re), psub(a.im, b.im)}; return r; }
static f2 f2mul(f2 a, f2 b)
{
    f2 r = {psub(pmul(a.re, b.re), pmul(a.im, b.im)), padd(pmul(a.re, b.im), pmul(a.im, b.re))};
    return r;
}
static int f2eq(f2 a, f2 b) { return a.re == b.re && a.im == b.im; }
static int f2ok(f2 a) { return a.re < P2_P && a.im < P2_P; }
static f2 f2scale(f2 a, uint64_t c) { f2 r = {pmul(a.re, c), pmul(a.im, c)}; return r; }
/* (a + b i)^-1 = (a - b i) / (a^2 + b^2); a^2 + b^2 != 0 for a nonzero element */
static f2 f2inv(f2 a)
{
    uint64_t nrm = padd(pmul(a.re, a.re), pmul(a.im, a.im));
    uint64_t ni = ppow(nrm, P2_P - 2);
    f2 r = {pmul(a.re, ni), pmul(psub(0, a.im), ni)};
    return r;
}

/* exported for the pins */
void orc2_mul(const uint64_t *a, const uint64_t *b, uint64_t *out)
{
    f2 x = {a[0], a[1]}, y = {b[0], b[1]}, r = f2mul(x, y);
    out[0] = r.re;
    out[1] = r.im;
}
void orc2_inv(const uint64_t *a, uint64_t *out)
{
    f2 x = {a[0], a[1]}, r = f2inv(x);
    out[0] = r.re;
    out[1] = r.im;
}

/* ------------------------------------------------------------------------ */
/* Multilinear extensions at points of F_{p^2}^v (Eq. (1), Sec. II-C).       */
/* ------------------------------------------------------------------------ */
static void chi_vector2(const f2 *z, int v, f2 *out)
{
    const f2 one = f2of(1);
    out[0] = one;
    for (int i = 0; i < v; i++) {
        size_t len = (size_t)1 << i;
        for (size_t y = len; y-- > 0;) {
            f2 e = out[y];
            out[2 * y] = f2mul(e, f2sub(one, z[i]));
            out[2 * y + 1] = f2mul(e, z[i]);
        }
    }
}

static f2 eq_points2(const f2 *a, const f2 *b, int v)
{
    /* eq(a, b) = prod_i (a_i b_i + (1 - a_i)(1 - b_i)) */
    const f2 one = f2of(1);
    f2 acc = one;
    for (int i = 0; i < v; i++)
        acc = f2mul(acc, f2add(f2mul(a[i], b[i]), f2mul(f2sub(one, a[i]), f2sub(one, b[i]))));
    return acc;
}

static int mle_int2(const int64_t *tab, int v, const f2 *z, f2 *out)
{
    size_t len = (size_t)1 << v;
    f2 *chi = (f2 *)malloc(len * sizeof(f2));
    if (!chi) return P2_E_NOMEM;
    chi_vector2(z, v, chi);
    f2 acc = f2of(0);
    for (size_t y = 0; y < len; y++) acc = f2add(acc, f2mul(f2int(tab[y]), chi[y]));
    free(chi);
    *out = acc;
    return P2_OK;
}

static int mle_f2(const f2 *tab, int v, const f2 *z, f2 *out)
{
    size_t len = (size_t)1 << v;
    f2 *chi = (f2 *)malloc(len * sizeof(f2));
    if (!chi) return P2_E_NOMEM;
    chi_vector2(z, v, chi);
    f2 acc = f2of(0);
    for (size_t y = 0; y < len; y++) acc = f2add(acc, f2mul(tab[y], chi[y]));
    free(chi);
    *out = acc;
    return P2_OK;
}

/* exported for the pins: MLE of an int64 table at a point (pairs re, im) */
int orc2_mle_int(const int64_t *tab, int v, const uint64_t *z, uint64_t *out)
{
    f2 zz[64], r;
    if (v > 64) return P2_E_INVAL;
    for (int i = 0; i < v; i++) {
        zz[i].re = z[2 * i];
        zz[i].im = z[2 * i + 1];
    }
    int rc = mle_int2(tab, v, zz, &r);
    out[0] = r.re;
    out[1] = r.im;
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Sum-check over F_{p^2} (Sec. II-D): the generic textbook prover and the   */
/* verifier's chain.                                                          */
/* ------------------------------------------------------------------------ */
typedef f2 (*summand2_fn)(const f2 *vals, const void *ctx);

/* ------------------------------------------------------------------------ */
/* Where the challenges come from: the F_p stream read in pairs (the          */
/* interactive protocol with the verifier's coins given), or the Fiat-Shamir */
/* transcript of ra_oracle_fs.c (each challenge a hash of what the prover     */
/* has sent).  Every challenge drawn is also logged, in order.                */
/* ------------------------------------------------------------------------ */
typedef struct {
    const uint64_t *chal; /* stream (fs == NULL) */
    int64_t nchal, *cursor;
    orc_fs *fs;
    f2 *log;
    int64_t nlog, cap;
    int err;
} chsrc;

static f2 src_draw(chsrc *src)
{
    f2 c = f2of(0);
    if (src->fs) {
        uint64_t w[2];
        orc_fs_draw(src->fs, w);
        c.re = w[0];
        c.im = w[1];
    } else if (*src->cursor < 0 || *src->cursor + 2 > src->nchal) {
        src->err = P2_E_CHALLENGES;
    } else {
        c.re = src->chal[*src->cursor];
        c.im = src->chal[*src->cursor + 1];
        if (!f2ok(c)) src->err = P2_E_CHALLENGES;
        *src->cursor += 2;
    }
    if (src->nlog < src->cap) src->log[src->nlog] = c;
    src->nlog++;
    return c;
}

static void src_absorb_bytes(chsrc *src, const uint8_t *b, uint32_t len)
{
    if (src->fs && orc_fs_absorb(src->fs, b, len) != 0) src->err = P2_E_INVAL;
}

static void src_absorb_f2(chsrc *src, const f2 *v, int count)
{
    for (int i = 0; i < count; i++) {
        uint8_t b[16];
        for (int j = 0; j < 8; j++) {
            b[j] = (uint8_t)(v[i].re >> (8 * j));
            b[8 + j] = (uint8_t)(v[i].im >> (8 * j));
        }
        src_absorb_bytes(src, b, 16);
    }
}

/*
 * The textbook sum-check prover (Sec. II-D) for sum_{x in {0,1}^v}
 * f(T_1(x), ..., T_q(x)) over multilinear tables.  Round j (x_j free,
 * x_1..x_{j-1} bound) sends g_j(X) at X = 0..deg, each table being lo + X
 * (hi - lo) in the free variable; the message is absorbed, the challenge
 * rho_j drawn, and every table bound at x_j = rho_j.  The tables are consumed.
 */
static void sumcheck_prove2_src(int v, int deg, int ntab, f2 **tabs, summand2_fn f, const void *fctx, chsrc *src,
                                f2 *rho_out, f2 *evals, f2 *finals)
{
    size_t size = (size_t)1 << v;
    f2 vals[8];
    for (int j = 0; j < v; j++) {
        size_t h = size / 2;
        f2 *g = evals + (size_t)j * (deg + 1);
        for (int X = 0; X <= deg; X++) {
            f2 acc = f2of(0);
            for (size_t i = 0; i < h; i++) {
                for (int q = 0; q < ntab; q++) {
                    f2 lo = tabs[q][i], hi = tabs[q][i + h];
                    vals[q] = f2add(lo, f2scale(f2sub(hi, lo), (uint64_t)X));
                }
                acc = f2add(acc, f(vals, fctx));
            }
            g[X] = acc;
        }
        src_absorb_f2(src, g, deg + 1);
        const f2 r = src_draw(src);
        rho_out[j] = r;
        for (int q = 0; q < ntab; q++)
            for (size_t i = 0; i < h; i++) tabs[q][i] = f2add(tabs[q][i], f2mul(r, f2sub(tabs[q][i + h], tabs[q][i])));
        size = h;
    }
    for (int q = 0; q < ntab; q++) finals[q] = tabs[q][0];
}

/* Lagrange interpolation through (0, e_0) .. (deg, e_deg) at x: the nodes
 * are integers, so the denominators are small integers of F_p. */
static f2 interp2(const f2 *e, int deg, f2 x)
{
    f2 acc = f2of(0);
    for (int i = 0; i <= deg; i++) {
        f2 num = f2of(1);
        int64_t den = 1;
        for (int j = 0; j <= deg; j++) {
            if (j == i) continue;
            num = f2mul(num, f2sub(x, f2int(j)));
            den *= (i - j);
        }
        acc = f2add(acc, f2mul(e[i], f2scale(num, ppow(pint(den), P2_P - 2))));
    }
    return acc;
}

static int sumcheck_chain2(int v, int deg, f2 claim, const f2 *evals, const f2 *rho, f2 *final_out)
{
    f2 cur = claim;
    for (int j = 0; j < v; j++) {
        const f2 *g = evals + (size_t)j * (deg + 1);
        for (int X = 0; X <= deg; X++)
            if (!f2ok(g[X])) return 0;
        if (!f2eq(f2add(g[0], g[1]), cur)) return 0;
        cur = interp2(g, deg, rho[j]);
    }
    *final_out = cur;
    return 1;
}

static f2 sm_matmul(const f2 *v, const void *ctx)
{
    (void)ctx;
    return f2mul(v[0], v[1]);
}
typedef struct { f2 mu; } range2_ctx;
static f2 sm_range(const f2 *v, const void *ctx)
{
    /* v = (eq(tau, .), W(plane) eq(r, x), b): eq b (b - 1) + mu G b */
    f2 mu = ((const range2_ctx *)ctx)->mu;
    f2 boole = f2mul(v[0], f2mul(v[2], f2sub(v[2], f2of(1))));
    return f2add(boole, f2mul(mu, f2mul(v[1], v[2])));
}
static f2 sm_relu(const f2 *v, const void *ctx)
{
    (void)ctx;
    return f2mul(v[0], f2sub(f2mul(v[1], v[1]), f2mul(v[2], v[2])));
}

static int ilog2x(int64_t x)
{
    if (x <= 0) return -1;
    int l = 0;
    while (((int64_t)1 << l) < x) l++;
    return (((int64_t)1 << l) == x) ? l : -1;
}

/* plane weights lambda_group 2^bit (reading of Alg. 1 steps 11-12, Sec. III-B) */
static void plane_weights2(f2 *W, int P, int s, int t, int relu, const f2 *lam)
{
    for (int q = 0; q < P; q++) W[q] = f2of(0);
    int q = 0;
    for (int b = 0; b < s; b++, q++) W[q] = f2scale(lam[0], pint((int64_t)1 << b));
    for (int b = 0; b < t + 2; b++, q++) W[q] = f2scale(lam[1], pint((int64_t)1 << b));
    if (relu)
        for (int b = 0; b < t + 2; b++, q++) W[q] = f2scale(lam[2], pint((int64_t)1 << b));
}

/* Scalars of a layer's transcript over F_{p^2}: each field element is two
 * words (re, im). */
typedef struct {
    int32_t t, P, log_p;
    int32_t n_mm_rounds, n_rs_rounds, n_zc_rounds;
    int64_t challenges_used; /* words of the F_p stream consumed (two per challenge) */
    f2 c0, a_star, b_star;
    f2 r_claim, rm_claim, y_claim, z_claim;
    f2 range_sum, bits_claim;
    f2 r_at, y_at;
} orc2_layer_info;

/* the challenges of a layer from the F_p stream at *cursor (two words each) */
static int take_challenges(const uint64_t *chal, int64_t nchal, int64_t *cursor, int64_t count, f2 *out)
{
    if (*cursor < 0 || *cursor + 2 * count > nchal) return P2_E_CHALLENGES;
    for (int64_t j = 0; j < count; j++) {
        out[j].re = chal[*cursor + 2 * j];
        out[j].im = chal[*cursor + 2 * j + 1];
        if (!f2ok(out[j])) return P2_E_CHALLENGES;
    }
    *cursor += 2 * count;
    return P2_OK;
}

/* the packed bit table: word x has bit q = plane q (P <= 64) */
static void pack_words(const uint8_t *bits, int64_t N, int P, uint64_t *words)
{
    for (int64_t x = 0; x < N; x++) {
        uint64_t w = 0;
        for (int q = 0; q < P && q < 64; q++) w |= (uint64_t)(bits[(size_t)q * N + x] & 1) << q;
        words[x] = w;
    }
}

static void absorb_header(chsrc *src, int64_t n, int64_t m, int64_t k, int s, int relu, int mode, int t, int P,
                          const uint8_t *pub, const uint8_t *root)
{
    const uint32_t h[8] = {(uint32_t)n, (uint32_t)m, (uint32_t)k, (uint32_t)s, (uint32_t)relu, (uint32_t)mode,
                           (uint32_t)t, (uint32_t)P};
    uint8_t b[32];
    for (int i = 0; i < 8; i++)
        for (int j = 0; j < 4; j++) b[4 * i + j] = (uint8_t)(h[i] >> (8 * j));
    src_absorb_bytes(src, b, 32);
    src_absorb_bytes(src, pub, 32);
    src_absorb_bytes(src, root, 32);
}

/*
 * One layer over F_{p^2}: the steps of orc_prove_layer (ra_oracle.c) with
 * every challenge-dependent value in F_{p^2}, the challenges drawn from `src`
 * at the points where the verifier sends them.  With a Fiat-Shamir source the
 * prover first absorbs the layer header, the caller's public digest `pub` and
 * the Merkle root of its witness tables; then each message (round values, the
 * final values and claims) before the challenge that follows it.  bits must
 * hold 128 N bytes; mm_evals 3 log m, rs_evals 4 (log P + log N), zc_evals
 * 4 log N elements.
 */
static int prove_layer_src(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu,
                           int mode, int t_in, chsrc *src, const uint8_t *pub, int64_t *C, int64_t *R, int64_t *Rm,
                           int64_t *Y, int64_t *Z, uint8_t *bits, f2 *mm_evals, f2 *rs_evals, f2 *zc_evals,
                           orc2_layer_info *info)
{
    int ln = ilog2x(n), lm = ilog2x(m), lk = ilog2x(k);
    if (ln < 0 || lm < 0 || lk < 0 || s < 1 || s > 30 || (mode != 0 && mode != 1)) return P2_E_INVAL;
    int64_t N = n * k;
    int lN = ln + lk;
    memset(info, 0, sizeof(*info));
    int t = 0, P = 1, lP = 0;
    int rc = orc_layer_witness(n, m, k, A, B, s, relu, mode, t_in, C, R, Rm, Y, Z, &t, &P, &lP);
    if (rc != 0) return rc;
    info->t = t;
    info->P = P;
    info->log_p = lP;
    info->n_mm_rounds = lm;
    info->n_rs_rounds = lP + lN;
    info->n_zc_rounds = relu ? lN : 0;
    int64_t need = ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    if (!src->fs && (*src->cursor < 0 || *src->cursor + 2 * need > src->nchal)) return P2_E_CHALLENGES;
    orc_fill_planes(bits, N, P, s, t, relu, R, Rm, Y);
    if (src->fs) {
        uint64_t *words = malloc(sizeof(uint64_t) * (size_t)N);
        uint8_t root[32];
        if (!words || P > 64) {
            free(words);
            return P2_E_INVAL;
        }
        pack_words(bits, N, P, words);
        rc = orc_witness_root(R, Rm, Y, Z, words, N, root);
        free(words);
        if (rc != 0) return P2_E_NOMEM;
        absorb_header(src, n, m, k, s, relu, mode, t, P, pub, root);
    }
    const int64_t draws0 = src->nlog;

    f2 *c = (f2 *)malloc(sizeof(f2) * (size_t)(need > 0 ? need : 1));
    if (!c) return P2_E_NOMEM;
    f2 *r1 = c, *r2 = c + ln, *rho = c + ln + lk, *lam = c + ln + lk + lm;
    f2 *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    for (int i = 0; i < ln; i++) r1[i] = src_draw(src);
    for (int i = 0; i < lk; i++) r2[i] = src_draw(src);

    /* Matrix sum-check (Eq. (4)): a(l) = sum_i chi_i(r1) A[i, l], b(l) = sum_j B[l, j] chi_j(r2). */
    f2 *chi1 = malloc(sizeof(f2) * (size_t)n), *chi2 = malloc(sizeof(f2) * (size_t)k);
    f2 *ta = malloc(sizeof(f2) * (size_t)m), *tb = malloc(sizeof(f2) * (size_t)m);
    f2 *r12 = malloc(sizeof(f2) * (size_t)(lN > 0 ? lN : 1));
    if (!chi1 || !chi2 || !ta || !tb || !r12) return P2_E_NOMEM;
    chi_vector2(r1, ln, chi1);
    chi_vector2(r2, lk, chi2);
    for (int64_t l = 0; l < m; l++) {
        f2 sa = f2of(0), sb = f2of(0);
        for (int64_t i = 0; i < n; i++) sa = f2add(sa, f2mul(chi1[i], f2int(A[i * m + l])));
        for (int64_t j = 0; j < k; j++) sb = f2add(sb, f2mul(f2int(B[l * k + j]), chi2[j]));
        ta[l] = sa;
        tb[l] = sb;
    }
    f2 c0 = f2of(0);
    for (int64_t l = 0; l < m; l++) c0 = f2add(c0, f2mul(ta[l], tb[l]));
    info->c0 = c0;
    {
        f2 *tabs[2] = {ta, tb}, fin[2];
        sumcheck_prove2_src(lm, 2, 2, tabs, sm_matmul, NULL, src, rho, mm_evals, fin);
        info->a_star = fin[0];
        info->b_star = fin[1];
    }
    free(ta);
    free(tb);

    /* Claims at (r1, r2). */
    for (int i = 0; i < ln; i++) r12[i] = r1[i];
    for (int i = 0; i < lk; i++) r12[ln + i] = r2[i];
    mle_int2(R, lN, r12, &info->r_claim);
    mle_int2(Rm, lN, r12, &info->rm_claim);
    mle_int2(Y, lN, r12, &info->y_claim);
    mle_int2(Z, lN, r12, &info->z_claim);
    {
        const f2 sent[6] = {info->a_star, info->b_star, info->r_claim, info->rm_claim, info->y_claim, info->z_claim};
        src_absorb_f2(src, sent, 6);
    }
    for (int i = 0; i < 4; i++) lam[i] = src_draw(src);
    for (int i = 0; i < lP; i++) tau_p[i] = src_draw(src);
    const f2 mu = lam[3];

    /* Concatenated range sum-check over b(plane, x), index plane N + x. */
    {
        int v = lP + lN;
        size_t L = (size_t)1 << v;
        f2 *teq = malloc(sizeof(f2) * L), *tg = malloc(sizeof(f2) * L), *tbits = malloc(sizeof(f2) * L);
        f2 *tau = malloc(sizeof(f2) * (size_t)(v > 0 ? v : 1)), *chix = malloc(sizeof(f2) * (size_t)N);
        f2 W[128];
        if (!teq || !tg || !tbits || !tau || !chix) return P2_E_NOMEM;
        for (int i = 0; i < lP; i++) tau[i] = tau_p[i];
        for (int i = 0; i < lN; i++) tau[lP + i] = r12[i];
        chi_vector2(tau, v, teq);
        chi_vector2(r12, lN, chix);
        plane_weights2(W, P, s, t, relu, lam);
        for (int q = 0; q < P; q++)
            for (int64_t x = 0; x < N; x++) {
                size_t idx = (size_t)q * N + x;
                tg[idx] = f2mul(W[q], chix[x]);
                tbits[idx] = f2of(bits[idx]);
            }
        f2 H = f2add(f2mul(lam[0], info->rm_claim),
                     f2mul(lam[1], f2add(info->r_claim, f2int((int64_t)1 << (t + 1)))));
        if (relu) H = f2add(H, f2mul(lam[2], info->y_claim));
        info->range_sum = f2mul(mu, H);
        range2_ctx rcx = {mu};
        f2 *tabs[3] = {teq, tg, tbits}, fin[3];
        sumcheck_prove2_src(v, 3, 3, tabs, sm_range, &rcx, src, sigma, rs_evals, fin);
        info->bits_claim = fin[2];
        src_absorb_f2(src, &info->bits_claim, 1);
        free(teq);
        free(tg);
        free(tbits);
        free(tau);

        /* ReLU zero-check (Eq. (6)) with the point (r1, r2). */
        if (relu) {
            f2 *tr = malloc(sizeof(f2) * (size_t)N), *ty = malloc(sizeof(f2) * (size_t)N);
            if (!tr || !ty) return P2_E_NOMEM;
            for (int64_t x = 0; x < N; x++) {
                tr[x] = f2int(R[x]);
                ty[x] = f2int(Y[x]);
            }
            f2 *tabs2[3] = {chix, tr, ty}, fin2[3];
            sumcheck_prove2_src(lN, 3, 3, tabs2, sm_relu, NULL, src, rho2, zc_evals, fin2);
            info->r_at = fin2[1];
            info->y_at = fin2[2];
            const f2 sent[2] = {info->r_at, info->y_at};
            src_absorb_f2(src, sent, 2);
            free(tr);
            free(ty);
        }
        free(chix);
    }
    info->challenges_used = 2 * (src->nlog - draws0);
    free(r12);
    free(chi1);
    free(chi2);
    free(c);
    return src->err;
}

/* The layer with the challenges read from the F_p stream in pairs (word
 * *cursor on). */
int orc2_prove_layer(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu, int mode,
                     int t_in, const uint64_t *chal, int64_t nchal, int64_t *cursor, int64_t *C, int64_t *R,
                     int64_t *Rm, int64_t *Y, int64_t *Z, uint8_t *bits, f2 *mm_evals, f2 *rs_evals, f2 *zc_evals,
                     orc2_layer_info *info)
{
    chsrc src = {chal, nchal, cursor, NULL, NULL, 0, 0, P2_OK};
    return prove_layer_src(n, m, k, A, B, s, relu, mode, t_in, &src, NULL, C, R, Rm, Y, Z, bits, mm_evals, rs_evals,
                           zc_evals, info);
}

/* The layer made non-interactive: the challenges from the Fiat-Shamir
 * transcript *fs (carried from layer to layer), pub the caller's 32-byte
 * digest of the public inputs.  drawn (optional, 2 (log n + log k + log m + 4
 * + 2 log P + log N (1 + relu)) words) receives every challenge drawn. */
int orc2_prove_layer_fs(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu,
                        int mode, int t_in, orc_fs *fs, const uint8_t *pub, int64_t *C, int64_t *R, int64_t *Rm,
                        int64_t *Y, int64_t *Z, uint8_t *bits, f2 *mm_evals, f2 *rs_evals, f2 *zc_evals,
                        orc2_layer_info *info, f2 *drawn, int64_t drawn_cap)
{
    int64_t cur = 0;
    chsrc src = {NULL, 0, &cur, fs, drawn, 0, drawn ? drawn_cap : 0, P2_OK};
    return prove_layer_src(n, m, k, A, B, s, relu, mode, t_in, &src, pub, C, R, Rm, Y, Z, bits, mm_evals, rs_evals,
                           zc_evals, info);
}

/*
 * Verify one layer over F_{p^2}: the checks of orc_verify_layer (ra_oracle.c)
 * with the same numbering, every transcript word a pair (re, im) in [0, p).
 */
int orc2_verify_layer(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, const int64_t *Z, int s,
                      int relu, int mode, const int64_t *R, const int64_t *Rm, const int64_t *Y,
                      const int64_t *bits, const f2 *mm_evals, const f2 *rs_evals, const f2 *zc_evals,
                      const orc2_layer_info *info, const uint64_t *chal, int64_t nchal, int64_t *cursor)
{
    int ln = ilog2x(n), lm = ilog2x(m), lk = ilog2x(k);
    if (ln < 0 || lm < 0 || lk < 0 || s < 1 || s > 30) return 13;
    int64_t N = n * k;
    int lN = ln + lk;
    int t = info->t;
    if (t < 0 || s + t + 3 > 61) return 12;
    int Q = s + (t + 2) + (relu ? (t + 2) : 0), P = 1, lP = 0;
    while (P < Q) { P *= 2; lP++; }
    if (info->P != P || P > 128) return 12;
    const f2 words[] = {info->c0, info->a_star, info->b_star, info->r_claim, info->rm_claim, info->y_claim,
                        info->z_claim, info->bits_claim, info->r_at, info->y_at, info->range_sum};
    for (int i = 0; i < 11; i++)
        if (!f2ok(words[i])) return 12;

    int64_t need = ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    f2 *c = (f2 *)malloc(sizeof(f2) * (size_t)(need > 0 ? need : 1));
    f2 *r12 = malloc(sizeof(f2) * (size_t)(lN > 0 ? lN : 1));
    if (!c || !r12) return 13;
    if (take_challenges(chal, nchal, cursor, need, c) != P2_OK) {
        free(c);
        free(r12);
        return 13;
    }
    const f2 *r1 = c, *r2 = c + ln, *rho = c + ln + lk, *lam = c + ln + lk + lm;
    const f2 mu = lam[3];
    const f2 *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    for (int i = 0; i < ln; i++) r12[i] = r1[i];
    for (int i = 0; i < lk; i++) r12[ln + i] = r2[i];
    int verdict = 0;
    f2 fin;

    /* 1-3: matrix chain, final a* b*, openings of a*, b* against A, B */
    if (!sumcheck_chain2(lm, 2, info->c0, mm_evals, rho, &fin)) { verdict = 1; goto done; }
    if (!f2eq(fin, f2mul(info->a_star, info->b_star))) { verdict = 2; goto done; }
    {
        f2 *pa = malloc(sizeof(f2) * (size_t)(ln + lm + 1)), *pb = malloc(sizeof(f2) * (size_t)(lm + lk + 1));
        for (int i = 0; i < ln; i++) pa[i] = r1[i];
        for (int i = 0; i < lm; i++) pa[ln + i] = rho[i];
        for (int i = 0; i < lm; i++) pb[i] = rho[i];
        for (int i = 0; i < lk; i++) pb[lm + i] = r2[i];
        f2 ea, eb;
        mle_int2(A, ln + lm, pa, &ea);
        mle_int2(B, lm + lk, pb, &eb);
        free(pa);
        free(pb);
        if (!f2eq(ea, info->a_star) || !f2eq(eb, info->b_star)) { verdict = 3; goto done; }
    }
    /* 4: rounding link C~ = 2^s R~ + Rm~ - 2^(s-1) (floor mode: no offset) */
    {
        f2 rhs = f2add(f2scale(info->r_claim, pint((int64_t)1 << s)), info->rm_claim);
        if (mode == 0) rhs = f2sub(rhs, f2int((int64_t)1 << (s - 1)));
        if (!f2eq(rhs, info->c0)) { verdict = 4; goto done; }
    }
    /* 5-7: range claimed sum, chain, final identity, bit-table opening */
    {
        f2 H = f2add(f2mul(lam[0], info->rm_claim), f2mul(lam[1], f2add(info->r_claim, f2int((int64_t)1 << (t + 1)))));
        if (relu) H = f2add(H, f2mul(lam[2], info->y_claim));
        H = f2mul(mu, H);
        if (!f2eq(H, info->range_sum)) { verdict = 5; goto done; }
        if (!sumcheck_chain2(lP + lN, 3, H, rs_evals, sigma, &fin)) { verdict = 5; goto done; }
        f2 W[128], wsig;
        plane_weights2(W, P, s, t, relu, lam);
        mle_f2(W, lP, sigma, &wsig);
        f2 eqp = eq_points2(tau_p, sigma, lP), eqx = eq_points2(r12, sigma + lP, lN);
        f2 bc = info->bits_claim;
        f2 expect = f2add(f2mul(f2mul(eqp, eqx), f2mul(bc, f2sub(bc, f2of(1)))), f2mul(mu, f2mul(f2mul(wsig, eqx), bc)));
        if (!f2eq(fin, expect)) { verdict = 6; goto done; }
        f2 eb;
        mle_int2(bits, lP + lN, sigma, &eb);
        if (!f2eq(eb, bc)) { verdict = 7; goto done; }
    }
    /* 8: openings of R, Rm, Y at (r1, r2) */
    {
        f2 er, erm, ey;
        mle_int2(R, lN, r12, &er);
        mle_int2(Rm, lN, r12, &erm);
        mle_int2(Y, lN, r12, &ey);
        if (!f2eq(er, info->r_claim) || !f2eq(erm, info->rm_claim) || !f2eq(ey, info->y_claim)) { verdict = 8; goto done; }
    }
    /* 9-10: ReLU chain from 0, final identity, openings at rho' */
    if (relu) {
        if (!sumcheck_chain2(lN, 3, f2of(0), zc_evals, rho2, &fin)) { verdict = 9; goto done; }
        f2 eqx = eq_points2(r12, rho2, lN);
        f2 expect = f2mul(eqx, f2sub(f2mul(info->r_at, info->r_at), f2mul(info->y_at, info->y_at)));
        if (!f2eq(fin, expect)) { verdict = 9; goto done; }
        f2 er, ey;
        mle_int2(R, lN, rho2, &er);
        mle_int2(Y, lN, rho2, &ey);
        if (!f2eq(er, info->r_at) || !f2eq(ey, info->y_at)) { verdict = 10; goto done; }
    }
    /* 11: output link 2 Z~ = R~ + Y~ (or Z~ = R~) and the opening of Z */
    {
        f2 ez;
        if (relu) {
            if (!f2eq(f2scale(info->z_claim, 2), f2add(info->r_claim, info->y_claim))) { verdict = 11; goto done; }
        } else if (!f2eq(info->z_claim, info->r_claim)) {
            verdict = 11;
            goto done;
        }
        mle_int2(Z, lN, r12, &ez);
        if (!f2eq(ez, info->z_claim)) { verdict = 11; goto done; }
    }
    (void)N;
done:
    free(c);
    free(r12);
    return verdict;
}

/*
 * Verify one layer made non-interactive: replay the prover's transcript
 * through *fs (header, pub, the Merkle root of the opened tables, then every
 * message in the prover's order) to recover the challenges, and run the
 * checks of orc2_verify_layer with them.  bits: the P x N planes (0 or 1).
 */
int orc2_verify_layer_fs(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, const int64_t *Z,
                         int s, int relu, int mode, const int64_t *R, const int64_t *Rm, const int64_t *Y,
                         const int64_t *bits, const f2 *mm_evals, const f2 *rs_evals, const f2 *zc_evals,
                         const orc2_layer_info *info, orc_fs *fs, const uint8_t *pub)
{
    int ln = ilog2x(n), lm = ilog2x(m), lk = ilog2x(k);
    if (ln < 0 || lm < 0 || lk < 0 || s < 1 || s > 30) return 13;
    int64_t N = n * k;
    int lN = ln + lk, t = info->t;
    if (t < 0 || s + t + 3 > 61) return 12;
    int Q = s + (t + 2) + (relu ? (t + 2) : 0), P = 1, lP = 0;
    while (P < Q) { P *= 2; lP++; }
    if (info->P != P || P > 64) return 12;
    uint64_t *words = malloc(sizeof(uint64_t) * (size_t)N);
    if (!words) return 13;
    for (int64_t x = 0; x < N; x++) {
        uint64_t w = 0;
        for (int q = 0; q < P; q++) {
            int64_t b = bits[(size_t)q * N + x];
            if (b != 0 && b != 1) {
                free(words);
                return 13;
            }
            w |= (uint64_t)b << q;
        }
        words[x] = w;
    }
    uint8_t root[32];
    int rc = orc_witness_root(R, Rm, Y, Z, words, N, root);
    free(words);
    if (rc != 0) return 13;
    int64_t need = ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    f2 *c = malloc(sizeof(f2) * (size_t)(need > 0 ? need : 1));
    uint64_t *chal = malloc(sizeof(uint64_t) * (size_t)(2 * need + 2));
    if (!c || !chal) {
        free(c);
        free(chal);
        return 13;
    }
    int64_t cur = 0;
    chsrc src = {NULL, 0, &cur, fs, c, 0, need, P2_OK};
    absorb_header(&src, n, m, k, s, relu, mode, t, P, pub, root);
    for (int i = 0; i < ln + lk; i++) src_draw(&src);
    for (int j = 0; j < lm; j++) {
        src_absorb_f2(&src, mm_evals + 3 * j, 3);
        src_draw(&src);
    }
    {
        const f2 sent[6] = {info->a_star, info->b_star, info->r_claim, info->rm_claim, info->y_claim, info->z_claim};
        src_absorb_f2(&src, sent, 6);
    }
    for (int i = 0; i < 4 + lP; i++) src_draw(&src);
    for (int j = 0; j < lP + lN; j++) {
        src_absorb_f2(&src, rs_evals + 4 * j, 4);
        src_draw(&src);
    }
    src_absorb_f2(&src, &info->bits_claim, 1);
    if (relu) {
        for (int j = 0; j < lN; j++) {
            src_absorb_f2(&src, zc_evals + 4 * j, 4);
            src_draw(&src);
        }
        const f2 sent[2] = {info->r_at, info->y_at};
        src_absorb_f2(&src, sent, 2);
    }
    int verdict = 13;
    if (src.err == P2_OK && src.nlog == need) {
        for (int64_t i = 0; i < need; i++) {
            chal[2 * i] = c[i].re;
            chal[2 * i + 1] = c[i].im;
        }
        int64_t cur2 = 0;
        verdict = orc2_verify_layer(n, m, k, A, B, Z, s, relu, mode, R, Rm, Y, bits, mm_evals, rs_evals, zc_evals,
                                    info, chal, 2 * need, &cur2);
    }
    free(c);
    free(chal);
    return verdict;
}

/* exported for the pins: the transcript's state, absorb and draw */
void orc2_fs_init(orc_fs *t, const uint8_t *domain) { orc_fs_init(t, domain); }
int orc2_fs_absorb(orc_fs *t, const uint8_t *m, uint32_t len) { return orc_fs_absorb(t, m, len); }
void orc2_fs_draw(orc_fs *t, uint64_t *out) { orc_fs_draw(t, out); }
