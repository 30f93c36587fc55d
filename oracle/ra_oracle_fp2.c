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

static void sumcheck_prove2(int v, int deg, int ntab, f2 **tabs, summand2_fn f, const void *fctx, const f2 *rho,
                            f2 *evals, f2 *finals)
{
    size_t size = (size_t)1 << v;
    f2 vals[8];
    for (int j = 0; j < v; j++) {
        size_t h = size / 2;
        for (int X = 0; X <= deg; X++) {
            f2 acc = f2of(0);
            for (size_t i = 0; i < h; i++) {
                for (int q = 0; q < ntab; q++) {
                    f2 lo = tabs[q][i], hi = tabs[q][i + h];
                    vals[q] = f2add(lo, f2scale(f2sub(hi, lo), (uint64_t)X));
                }
                acc = f2add(acc, f(vals, fctx));
            }
            evals[(size_t)j * (deg + 1) + X] = acc;
        }
        for (int q = 0; q < ntab; q++)
            for (size_t i = 0; i < h; i++)
                tabs[q][i] = f2add(tabs[q][i], f2mul(rho[j], f2sub(tabs[q][i + h], tabs[q][i])));
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

/*
 * Prove one layer over F_{p^2}: the steps of orc_prove_layer (ra_oracle.c)
 * with every challenge-dependent value in F_{p^2}.  bits must hold 128 N
 * bytes; mm_evals 3 log m, rs_evals 4 (log P + log N), zc_evals 4 log N
 * elements.
 */
int orc2_prove_layer(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu, int mode,
                     int t_in, const uint64_t *chal, int64_t nchal, int64_t *cursor, int64_t *C, int64_t *R,
                     int64_t *Rm, int64_t *Y, int64_t *Z, uint8_t *bits, f2 *mm_evals, f2 *rs_evals, f2 *zc_evals,
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
    f2 *c = (f2 *)malloc(sizeof(f2) * (size_t)(need > 0 ? need : 1));
    if (!c) return P2_E_NOMEM;
    int64_t cur0 = *cursor;
    if ((rc = take_challenges(chal, nchal, cursor, need, c)) != P2_OK) {
        free(c);
        return rc;
    }
    info->challenges_used = *cursor - cur0;
    const f2 *r1 = c, *r2 = c + ln, *rho = c + ln + lk, *lam = c + ln + lk + lm;
    const f2 mu = lam[3];
    const f2 *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;

    orc_fill_planes(bits, N, P, s, t, relu, R, Rm, Y);

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
        sumcheck_prove2(lm, 2, 2, tabs, sm_matmul, NULL, rho, mm_evals, fin);
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
        sumcheck_prove2(v, 3, 3, tabs, sm_range, &rcx, sigma, rs_evals, fin);
        info->bits_claim = fin[2];
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
            sumcheck_prove2(lN, 3, 3, tabs2, sm_relu, NULL, rho2, zc_evals, fin2);
            info->r_at = fin2[1];
            info->y_at = fin2[2];
            free(tr);
            free(ty);
        }
        free(chix);
    }
    free(r12);
    free(chi1);
    free(chi2);
    free(c);
    return P2_OK;
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
