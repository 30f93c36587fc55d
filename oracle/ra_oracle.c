/*
 * ra_oracle.c -- plain, slow CPU oracle for one layer of the Range-Arithmetic
 * protocol (matrix multiplication + fixed-point rounding + optional ReLU).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file.  It exists so that tests, the smoke check and the CPU
 * baseline of the benchmark can compare the GPU prover against an independent
 * implementation written straight from the paper's definitions.  It shares no
 * code, header, table or constant with the GPU path.
 *
 * Style: every field operation is a 128-bit integer product or sum followed by
 * "% p"; every multilinear extension is the Lagrange-basis sum of Eq. (1) /
 * Sec. II-C; every sum-check is the textbook round-by-round algorithm of
 * Sec. II-D over fully materialised tables (no blocking, fusion or reordering).
 *
 * Field: p = 2^61 - 1 (the paper fixes no prime; Sec. II-F asks for > 128 bits,
 * the reduced field is a stated reading).  Elements are canonical in [0, p);
 * the symmetric residue system of Definition II.1 is only used to lift values
 * back to signed integers.
 *
 * Conventions (readings of passages the paper leaves open):
 *  - A table of 2^v entries is a function on {0,1}^v; index bit v-1 (the MSB)
 *    is the first variable x_1 (worked example f_A([0,0],[1,0]) = a_{0,2},
 *    Sec. III-A-1).  Matrices are row-major, row bits before column bits.
 *  - Sum-check binds x_1 first; round j sends the round polynomial's values at
 *    X = 0..d (Sec. II-D).
 *  - Rounding is the operator R(x) of Sec. II-A with the mathematical floor
 *    modulo (the only reading under which the discarded part lies in
 *    [-2^(s-1), 2^(s-1)) as Sec. III-A-2 states).  A floor mode (no 2^(s-1)
 *    offset) is provided as well.
 *  - The two range conditions of Alg. 1 steps 11-12 and the Y >= 0 condition
 *    of Sec. III-B are proven by one concatenated bit table per layer whose
 *    booleanity and recomposition are proven by one sum-check.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define ORC_P ((uint64_t)0x1FFFFFFFFFFFFFFFULL) /* 2^61 - 1 */

enum {
    ORC_OK = 0,
    ORC_E_INVAL = -1,
    ORC_E_FIELD_TOO_SMALL = -3,
    ORC_E_RANGE = -4,
    ORC_E_CHALLENGES = -5,
    ORC_E_NOMEM = -10
};

/* ------------------------------------------------------------------------ */
/* Field F_p (Definition II.1).                                              */
/* ------------------------------------------------------------------------ */
static uint64_t fadd(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a + b) % ORC_P); }
static uint64_t fsub(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a + ORC_P - b) % ORC_P); }
static uint64_t fmul(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a * b) % ORC_P); }
static uint64_t fint(int64_t z)
{
    /* the field element congruent to the integer z */
    int64_t r = z % (int64_t)ORC_P;
    if (r < 0) r += (int64_t)ORC_P;
    return (uint64_t)r;
}
static uint64_t fpow2(int e) { return fint((int64_t)1 << e); }

/* ------------------------------------------------------------------------ */
/* Multilinear extensions (Definition II.2, Eq. (1); Lagrange basis chi of   */
/* Sec. II-C).                                                               */
/* ------------------------------------------------------------------------ */

/* chi_y(z) = prod_{i=1..v} (z_i y_i + (1 - z_i)(1 - y_i)), y_1 = MSB of y. */
static uint64_t chi_at(const uint64_t *z, int v, uint64_t y)
{
    uint64_t acc = 1;
    for (int i = 0; i < v; i++) {
        int yi = (int)((y >> (v - 1 - i)) & 1);
        acc = fmul(acc, yi ? z[i] : fsub(1, z[i]));
    }
    return acc;
}

/* All 2^v basis values.  Built variable by variable: after the first i
 * variables the vector holds chi over {0,1}^i; appending x_{i+1} splits every
 * entry into its (1 - z) and z parts.  The result equals chi_at for every y
 * (a test checks this against Eq. (1) directly). */
static int chi_vector(const uint64_t *z, int v, uint64_t *out)
{
    out[0] = 1;
    for (int i = 0; i < v; i++) {
        size_t len = (size_t)1 << i;
        for (size_t y = len; y-- > 0;) {
            uint64_t e = out[y];
            out[2 * y] = fmul(e, fsub(1, z[i]));
            out[2 * y + 1] = fmul(e, z[i]);
        }
    }
    return ORC_OK;
}

/* e~(z) = sum_y e(y) chi_y(z) for a table of field elements. */
static int mle_field(const uint64_t *tab, int v, const uint64_t *z, uint64_t *out)
{
    size_t len = (size_t)1 << v;
    uint64_t *chi = (uint64_t *)malloc(len * sizeof(uint64_t));
    if (!chi) return ORC_E_NOMEM;
    chi_vector(z, v, chi);
    uint64_t acc = 0;
    for (size_t y = 0; y < len; y++) acc = fadd(acc, fmul(tab[y], chi[y]));
    free(chi);
    *out = acc;
    return ORC_OK;
}

/* Same for a table of signed integers embedded in F_p. */
static int mle_int(const int64_t *tab, int v, const uint64_t *z, uint64_t *out)
{
    size_t len = (size_t)1 << v;
    uint64_t *chi = (uint64_t *)malloc(len * sizeof(uint64_t));
    if (!chi) return ORC_E_NOMEM;
    chi_vector(z, v, chi);
    uint64_t acc = 0;
    for (size_t y = 0; y < len; y++) acc = fadd(acc, fmul(fint(tab[y]), chi[y]));
    free(chi);
    *out = acc;
    return ORC_OK;
}

/* Exported for tests: MLE of an int64 table, of a field table, and one chi. */
int orc_mle_int(const int64_t *tab, int v, const uint64_t *z, uint64_t *out) { return mle_int(tab, v, z, out); }
int orc_mle_field(const uint64_t *tab, int v, const uint64_t *z, uint64_t *out) { return mle_field(tab, v, z, out); }
uint64_t orc_chi_at(const uint64_t *z, int v, uint64_t y) { return chi_at(z, v, y); }
int orc_chi_vector(const uint64_t *z, int v, uint64_t *out) { return chi_vector(z, v, out); }
uint64_t orc_fmul(uint64_t a, uint64_t b) { return fmul(a, b); }
uint64_t orc_fadd(uint64_t a, uint64_t b) { return fadd(a, b); }
uint64_t orc_fsub(uint64_t a, uint64_t b) { return fsub(a, b); }
uint64_t orc_fint(int64_t z) { return fint(z); }

/* ------------------------------------------------------------------------ */
/* Generic sum-check prover (Sec. II-D).                                     */
/* ------------------------------------------------------------------------ */

/* The summand is a polynomial in the values of ntab multilinear tables. */
typedef uint64_t (*summand_fn)(const uint64_t *vals, const void *ctx);

/*
 * Proves sum_{x in {0,1}^v} f(T_1(x), ..., T_q(x)) for multilinear T_i.
 * Round j (x_j free, x_1..x_{j-1} bound to the earlier challenges) sends
 *     g_j(X) = sum_{x' in {0,1}^{v-j}} f(T(rho_1..rho_{j-1}, X, x'))
 * at X = 0..deg.  Each table restricted to the free variable is linear in X,
 * so its value at X is lo + X (hi - lo).  After the round every table is
 * bound at x_j = rho_j, which halves it.  The tables are consumed.
 */
static void sumcheck_prove(int v, int deg, int ntab, uint64_t **tabs, summand_fn f, const void *fctx,
                           const uint64_t *rho, uint64_t *evals, uint64_t *finals)
{
    size_t size = (size_t)1 << v;
    uint64_t vals[8];
    for (int j = 0; j < v; j++) {
        size_t h = size / 2;
        for (int X = 0; X <= deg; X++) {
            uint64_t acc = 0;
            for (size_t i = 0; i < h; i++) {
                for (int q = 0; q < ntab; q++) {
                    uint64_t lo = tabs[q][i], hi = tabs[q][i + h];
                    vals[q] = fadd(lo, fmul(fint(X), fsub(hi, lo)));
                }
                acc = fadd(acc, f(vals, fctx));
            }
            evals[(size_t)j * (deg + 1) + X] = acc;
        }
        for (int q = 0; q < ntab; q++)
            for (size_t i = 0; i < h; i++)
                tabs[q][i] = fadd(tabs[q][i], fmul(rho[j], fsub(tabs[q][i + h], tabs[q][i])));
        size = h;
    }
    for (int q = 0; q < ntab; q++) finals[q] = tabs[q][0];
}

/* Evaluate the polynomial of degree <= deg through (0, e_0), ..., (deg, e_deg)
 * at x, by the Lagrange interpolation formula. */
static uint64_t inv_small(int64_t d)
{
    /* inverse of a small nonzero integer by Fermat: d^(p-2) */
    uint64_t base = fint(d), r = 1, e = ORC_P - 2;
    while (e) {
        if (e & 1) r = fmul(r, base);
        base = fmul(base, base);
        e >>= 1;
    }
    return r;
}
static uint64_t interp(const uint64_t *e, int deg, uint64_t x)
{
    uint64_t acc = 0;
    for (int i = 0; i <= deg; i++) {
        uint64_t num = 1;
        int64_t den = 1;
        for (int j = 0; j <= deg; j++) {
            if (j == i) continue;
            num = fmul(num, fsub(x, fint(j)));
            den *= (i - j);
        }
        acc = fadd(acc, fmul(e[i], fmul(num, inv_small(den))));
    }
    return acc;
}
uint64_t orc_interp(const uint64_t *e, int deg, uint64_t x) { return interp(e, deg, x); }

/* Sum-check verifier chain (Sec. II-D): g_1(0) + g_1(1) = claim;
 * g_j(0) + g_j(1) = g_{j-1}(rho_{j-1}); returns g_v(rho_v) in *final_out. */
static int sumcheck_chain(int v, int deg, uint64_t claim, const uint64_t *evals, const uint64_t *rho,
                          uint64_t *final_out)
{
    uint64_t cur = claim;
    for (int j = 0; j < v; j++) {
        const uint64_t *g = evals + (size_t)j * (deg + 1);
        for (int X = 0; X <= deg; X++)
            if (g[X] >= ORC_P) return 0;
        if (fadd(g[0], g[1]) != cur) return 0;
        cur = interp(g, deg, rho[j]);
    }
    *final_out = cur;
    return 1;
}

/* Summands of the three sum-check instances of a layer. */
static uint64_t summand_matmul(const uint64_t *v, const void *ctx)
{
    (void)ctx; /* gamma(l) = a~(r1, l) b~(l, r2), Eq. (4) */
    return fmul(v[0], v[1]);
}
typedef struct { uint64_t mu; } range_ctx;
static uint64_t summand_range(const uint64_t *v, const void *ctx)
{
    /* v = (eq(tau, .), W(plane) eq(r, x), b):  eq b (b - 1) + mu G b */
    uint64_t mu = ((const range_ctx *)ctx)->mu;
    uint64_t boole = fmul(v[0], fmul(v[2], fsub(v[2], 1)));
    uint64_t recomp = fmul(mu, fmul(v[1], v[2]));
    return fadd(boole, recomp);
}
static uint64_t summand_relu(const uint64_t *v, const void *ctx)
{
    (void)ctx; /* I~(s, x) (a~^2(x) - y~^2(x)), Eq. (6) */
    return fmul(v[0], fsub(fmul(v[1], v[1]), fmul(v[2], v[2])));
}

/* ------------------------------------------------------------------------ */
/* Layer protocol.                                                           */
/* ------------------------------------------------------------------------ */

static int ilog2_exact(int64_t x)
{
    if (x <= 0) return -1;
    int l = 0;
    while (((int64_t)1 << l) < x) l++;
    return (((int64_t)1 << l) == x) ? l : -1;
}

/* floor division and floor modulo by 2^s (mathematical, not C truncation) */
static int64_t floor_div_pow2(int64_t x, int s)
{
    int64_t d = (int64_t)1 << s;
    int64_t q = x / d;
    if ((x % d) != 0 && x < 0) q -= 1;
    return q;
}

/* Number of planes per group and total (reading of Alg. 1 steps 11-12 and
 * Sec. III-B): s bits of the shifted remainder, t+2 bits of R + 2^(t+1),
 * t+2 bits of Y = |R| when the layer has a ReLU. */
int orc_plane_count(int s, int t, int relu) { return s + (t + 2) + (relu ? (t + 2) : 0); }

/* Output sizes of a layer's transcript, so a caller can size its buffers. */
typedef struct {
    int32_t t, P, log_p;
    int32_t n_mm_rounds, n_rs_rounds, n_zc_rounds;
    int64_t challenges_used;
    uint64_t c0, a_star, b_star;
    uint64_t r_claim, rm_claim, y_claim, z_claim;
    uint64_t range_sum, bits_claim;
    uint64_t r_at, y_at;
} orc_layer_info;

/* Fill the bit-plane table (plane-major, one byte per bit, P x N). */
static void fill_planes(uint8_t *bits, int64_t N, int P, int s, int t, int relu, const int64_t *R,
                        const int64_t *Rm, const int64_t *Y)
{
    memset(bits, 0, (size_t)P * (size_t)N);
    for (int64_t x = 0; x < N; x++) {
        int q = 0;
        for (int b = 0; b < s; b++, q++) bits[(size_t)q * N + x] = (uint8_t)((Rm[x] >> b) & 1);
        int64_t shifted = R[x] + ((int64_t)1 << (t + 1));
        for (int b = 0; b < t + 2; b++, q++) bits[(size_t)q * N + x] = (uint8_t)((shifted >> b) & 1);
        if (relu)
            for (int b = 0; b < t + 2; b++, q++) bits[(size_t)q * N + x] = (uint8_t)((Y[x] >> b) & 1);
    }
}

/* Weight of each plane in the recomposition (lambda_group * 2^bit). */
static void plane_weights(uint64_t *W, int P, int s, int t, int relu, const uint64_t *lam)
{
    for (int q = 0; q < P; q++) W[q] = 0;
    int q = 0;
    for (int b = 0; b < s; b++, q++) W[q] = fmul(lam[0], fpow2(b));
    for (int b = 0; b < t + 2; b++, q++) W[q] = fmul(lam[1], fpow2(b));
    if (relu)
        for (int b = 0; b < t + 2; b++, q++) W[q] = fmul(lam[2], fpow2(b));
}

/*
 * The layer's witness (Alg. 1 steps 2 and 9, Sec. III-B) and its range
 * parameters: C = A B over the integers, R = the rounding of C (mode 0: the
 * operator of Sec. II-A; 1: floor), the shifted remainder Rm, Y = |R|, the
 * output Z, the least t >= 0 with -2^(t+1) <= R < 2^(t+1) (t_in >= 0: that
 * t, checked), the field guard s + t + 3 <= 61 (Theorem A.1) and the plane
 * count P (a power of two).  Shared by the prover over F_p below and the one
 * over F_{p^2} (ra_oracle_fp2.c): the witness does not depend on the field.
 */
int orc_layer_witness(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu,
                      int mode, int t_in, int64_t *C, int64_t *R, int64_t *Rm, int64_t *Y, int64_t *Z, int *t_out,
                      int *P_out, int *lP_out)
{
    int64_t N = n * k;
    /* Witness: C = A B over the integers (Alg. 1 step 2). */
    for (int64_t i = 0; i < n; i++)
        for (int64_t j = 0; j < k; j++) C[i * k + j] = 0;
    for (int64_t i = 0; i < n; i++)
        for (int64_t l = 0; l < m; l++) {
            int64_t a = A[i * m + l];
            for (int64_t j = 0; j < k; j++) C[i * k + j] += a * B[l * k + j];
        }

    /* Rounding (Sec. II-A; Alg. 1 step 9) and ReLU (Sec. III-B). */
    int64_t half = mode == 0 ? ((int64_t)1 << (s - 1)) : 0;
    for (int64_t x = 0; x < N; x++) {
        R[x] = floor_div_pow2(C[x] + half, s);
        Rm[x] = C[x] + half - R[x] * ((int64_t)1 << s); /* E + 2^(s-1), in [0, 2^s) */
        Y[x] = R[x] < 0 ? -R[x] : R[x];
        Z[x] = relu ? (R[x] + Y[x]) / 2 : R[x];
    }

    /* t: least t >= 0 with -2^(t+1) <= R < 2^(t+1) (Condition 2 of Theorem A.1). */
    int t;
    if (t_in < 0) {
        t = 0;
        for (int64_t x = 0; x < N; x++)
            while (!(R[x] >= -((int64_t)1 << (t + 1)) && R[x] < ((int64_t)1 << (t + 1)))) t++;
    } else {
        t = t_in;
        if (t > 60) return ORC_E_RANGE;
        for (int64_t x = 0; x < N; x++)
            if (!(R[x] >= -((int64_t)1 << (t + 1)) && R[x] < ((int64_t)1 << (t + 1)))) return ORC_E_RANGE;
    }
    /* Field guard: p must have at least s + t + 3 bits (Theorem A.1). */
    if (s + t + 3 > 61) return ORC_E_FIELD_TOO_SMALL;
    int Q = orc_plane_count(s, t, relu);
    int P = 1, lP = 0;
    while (P < Q) { P *= 2; lP++; }
    if (P > 128) return ORC_E_RANGE;
    *t_out = t;
    *P_out = P;
    *lP_out = lP;
    return ORC_OK;
}

/* The bit table of a layer, exported for the F_{p^2} prover. */
void orc_fill_planes(uint8_t *bits, int64_t N, int P, int s, int t, int relu, const int64_t *R, const int64_t *Rm,
                     const int64_t *Y)
{
    fill_planes(bits, N, P, s, t, relu, R, Rm, Y);
}

/*
 * Prove one layer.  Inputs: A (n x m), B (m x k) as int64 (values that fit the
 * layer's dtypes), s fractional bits, relu flag, mode (0 = rounding operator
 * of Sec. II-A, 1 = floor), t_in (< 0: least t that holds R; else given).
 * The challenge stream chal[0..nchal) is consumed from *cursor in this order:
 *   r1 (log n), r2 (log k), rho (log m), lambda1..3, mu, tau_p (log P),
 *   sigma (log P + log N), and with ReLU rho' (log N).
 * Outputs: C, R, Rm, Y, Z (n*k each), bits (P*N bytes, plane-major; the buffer
 * must hold 128*N bytes), transcript arrays mm_evals (3 per round), rs_evals
 * (4 per round), zc_evals (4 per round) and the scalars in *info.
 */
int orc_prove_layer(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, int s, int relu,
                    int mode, int t_in, const uint64_t *chal, int64_t nchal, int64_t *cursor, int64_t *C,
                    int64_t *R, int64_t *Rm, int64_t *Y, int64_t *Z, uint8_t *bits, uint64_t *mm_evals,
                    uint64_t *rs_evals, uint64_t *zc_evals, orc_layer_info *info)
{
    int ln = ilog2_exact(n), lm = ilog2_exact(m), lk = ilog2_exact(k);
    if (ln < 0 || lm < 0 || lk < 0 || s < 1 || s > 30 || (mode != 0 && mode != 1)) return ORC_E_INVAL;
    int64_t N = n * k;
    int lN = ln + lk;
    memset(info, 0, sizeof(*info));

    int t = 0, P = 1, lP = 0;
    {
        int rc = orc_layer_witness(n, m, k, A, B, s, relu, mode, t_in, C, R, Rm, Y, Z, &t, &P, &lP);
        if (rc != ORC_OK) return rc;
    }
    info->t = t;
    info->P = P;
    info->log_p = lP;
    info->n_mm_rounds = lm;
    info->n_rs_rounds = lP + lN;
    info->n_zc_rounds = relu ? lN : 0;

    int64_t need = ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    if (*cursor < 0 || *cursor + need > nchal) return ORC_E_CHALLENGES;
    const uint64_t *c = chal + *cursor;
    const uint64_t *r1 = c, *r2 = c + ln, *rho = c + ln + lk, *lam = c + ln + lk + lm;
    uint64_t mu = lam[3];
    const uint64_t *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    for (int64_t i = 0; i < need; i++)
        if (c[i] >= ORC_P) return ORC_E_CHALLENGES;
    *cursor += need;
    info->challenges_used = need;

    fill_planes(bits, N, P, s, t, relu, R, Rm, Y);

    /* Matrix multiplication sum-check (Sec. III-A-1, Eq. (4); Alg. 1 step 6):
     * gamma(l) = a~(r1, l) b~(l, r2) with a~(r1, .) = sum_i chi_i(r1) A[i, .]
     * and b~(., r2) = sum_j B[., j] chi_j(r2). */
    uint64_t *chi1 = malloc(sizeof(uint64_t) * (size_t)n);
    uint64_t *chi2 = malloc(sizeof(uint64_t) * (size_t)k);
    uint64_t *ta = malloc(sizeof(uint64_t) * (size_t)m);
    uint64_t *tb = malloc(sizeof(uint64_t) * (size_t)m);
    if (!chi1 || !chi2 || !ta || !tb) return ORC_E_NOMEM;
    chi_vector(r1, ln, chi1);
    chi_vector(r2, lk, chi2);
    for (int64_t l = 0; l < m; l++) {
        uint64_t sa = 0, sb = 0;
        for (int64_t i = 0; i < n; i++) sa = fadd(sa, fmul(chi1[i], fint(A[i * m + l])));
        for (int64_t j = 0; j < k; j++) sb = fadd(sb, fmul(fint(B[l * k + j]), chi2[j]));
        ta[l] = sa;
        tb[l] = sb;
    }
    uint64_t c0 = 0;
    for (int64_t l = 0; l < m; l++) c0 = fadd(c0, fmul(ta[l], tb[l]));
    info->c0 = c0;
    {
        uint64_t *tabs[2] = {ta, tb}, fin[2];
        sumcheck_prove(lm, 2, 2, tabs, summand_matmul, NULL, rho, mm_evals, fin);
        info->a_star = fin[0];
        info->b_star = fin[1];
    }
    free(ta);
    free(tb);

    /* Claims on the rounded output, its remainder, |R| and the layer output,
     * all at the point (r1, r2). */
    uint64_t *r12 = malloc(sizeof(uint64_t) * (size_t)(lN > 0 ? lN : 1));
    for (int i = 0; i < ln; i++) r12[i] = r1[i];
    for (int i = 0; i < lk; i++) r12[ln + i] = r2[i];
    mle_int(R, lN, r12, &info->r_claim);
    mle_int(Rm, lN, r12, &info->rm_claim);
    mle_int(Y, lN, r12, &info->y_claim);
    mle_int(Z, lN, r12, &info->z_claim);

    /* Concatenated range sum-check over the bit table b(plane, x), index
     * plane * N + x.  Booleanity with eq(tau, .), tau = (tau_p, r1, r2), plus
     * mu times the recomposition sum_plane W(plane) b(plane, x) at (r1, r2). */
    {
        int v = lP + lN;
        size_t L = (size_t)1 << v;
        uint64_t *teq = malloc(sizeof(uint64_t) * L);
        uint64_t *tg = malloc(sizeof(uint64_t) * L);
        uint64_t *tbits = malloc(sizeof(uint64_t) * L);
        uint64_t *tau = malloc(sizeof(uint64_t) * (size_t)v);
        uint64_t *chix = malloc(sizeof(uint64_t) * (size_t)N);
        uint64_t W[128];
        if (!teq || !tg || !tbits || !tau || !chix) return ORC_E_NOMEM;
        for (int i = 0; i < lP; i++) tau[i] = tau_p[i];
        for (int i = 0; i < lN; i++) tau[lP + i] = r12[i];
        chi_vector(tau, v, teq);
        chi_vector(r12, lN, chix);
        plane_weights(W, P, s, t, relu, lam);
        for (int q = 0; q < P; q++)
            for (int64_t x = 0; x < N; x++) {
                size_t idx = (size_t)q * N + x;
                tg[idx] = fmul(W[q], chix[x]);
                tbits[idx] = bits[idx];
            }
        /* claimed sum: mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~) at (r1, r2) */
        uint64_t H = fadd(fmul(lam[0], info->rm_claim), fmul(lam[1], fadd(info->r_claim, fpow2(t + 1))));
        if (relu) H = fadd(H, fmul(lam[2], info->y_claim));
        info->range_sum = fmul(mu, H);
        range_ctx rc = {mu};
        uint64_t *tabs[3] = {teq, tg, tbits}, fin[3];
        sumcheck_prove(v, 3, 3, tabs, summand_range, &rc, sigma, rs_evals, fin);
        info->bits_claim = fin[2];
        free(teq);
        free(tg);
        free(tbits);
        free(tau);

        /* ReLU square-equality zero-check (Sec. III-B, Eq. (6)) with s = (r1, r2). */
        if (relu) {
            uint64_t *tr = malloc(sizeof(uint64_t) * (size_t)N);
            uint64_t *ty = malloc(sizeof(uint64_t) * (size_t)N);
            if (!tr || !ty) return ORC_E_NOMEM;
            for (int64_t x = 0; x < N; x++) {
                tr[x] = fint(R[x]);
                ty[x] = fint(Y[x]);
            }
            uint64_t *tabs2[3] = {chix, tr, ty}, fin2[3];
            sumcheck_prove(lN, 3, 3, tabs2, summand_relu, NULL, rho2, zc_evals, fin2);
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
    return ORC_OK;
}

/*
 * Verify one layer (Sec. IV).  The verifier is given the public A, B, the
 * public output Z, the transcript, and -- in place of the paper's commitments
 * -- the opened tables R, Rm, Y and the bit table, from which it evaluates
 * multilinear extensions itself.  Returns 0 on accept, else the number of the
 * first failing check:
 *   1 matmul chain, 2 matmul final a* b*, 3 a* / b* against A / B,
 *   4 rounding link c0 = 2^s R~ + Rm~ - 2^(s-1), 5 range chain,
 *   6 range final identity, 7 bit-table opening, 8 R / Rm / Y openings,
 *   9 ReLU chain + final identity, 10 ReLU openings, 11 output link
 *   2 Z~ = R~ + Y~ (or Z~ = R~) and Z opening, 12 parameters (field guard,
 *   plane count, transcript words >= p), 13 malformed call.
 * The opened bit table is taken as arbitrary integers (P x N, plane-major):
 * booleanity is not inspected entry by entry but proven by the sum-check,
 * as it would be against a commitment.
 */
int orc_verify_layer(int64_t n, int64_t m, int64_t k, const int64_t *A, const int64_t *B, const int64_t *Z,
                     int s, int relu, int mode, const int64_t *R, const int64_t *Rm, const int64_t *Y,
                     const int64_t *bits, const uint64_t *mm_evals, const uint64_t *rs_evals,
                     const uint64_t *zc_evals, const orc_layer_info *info, const uint64_t *chal, int64_t nchal,
                     int64_t *cursor)
{
    int ln = ilog2_exact(n), lm = ilog2_exact(m), lk = ilog2_exact(k);
    if (ln < 0 || lm < 0 || lk < 0 || s < 1 || s > 30) return 13;
    int64_t N = n * k;
    int lN = ln + lk;
    int t = info->t;
    if (t < 0 || s + t + 3 > 61) return 12;
    int Q = orc_plane_count(s, t, relu), P = 1, lP = 0;
    while (P < Q) { P *= 2; lP++; }
    if (info->P != P || P > 128) return 12;
    const uint64_t words[] = {info->c0, info->a_star, info->b_star, info->r_claim, info->rm_claim,
                              info->y_claim, info->z_claim, info->bits_claim, info->r_at, info->y_at};
    for (int i = 0; i < 10; i++)
        if (words[i] >= ORC_P) return 12;

    int64_t need = ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    if (*cursor < 0 || *cursor + need > nchal) return 13;
    const uint64_t *c = chal + *cursor;
    const uint64_t *r1 = c, *r2 = c + ln, *rho = c + ln + lk, *lam = c + ln + lk + lm;
    uint64_t mu = lam[3];
    const uint64_t *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    *cursor += need;

    uint64_t *r12 = malloc(sizeof(uint64_t) * (size_t)(lN > 0 ? lN : 1));
    for (int i = 0; i < ln; i++) r12[i] = r1[i];
    for (int i = 0; i < lk; i++) r12[ln + i] = r2[i];
    int verdict = 0;

    /* 1-2: matrix multiplication sum-check chain */
    uint64_t fin;
    if (!sumcheck_chain(lm, 2, info->c0, mm_evals, rho, &fin)) { verdict = 1; goto done; }
    if (fin != fmul(info->a_star, info->b_star)) { verdict = 2; goto done; }
    /* 3: a* = A~(r1, rho), b* = B~(rho, r2) from the public matrices */
    {
        uint64_t *pa = malloc(sizeof(uint64_t) * (size_t)(ln + lm + 1));
        uint64_t *pb = malloc(sizeof(uint64_t) * (size_t)(lm + lk + 1));
        for (int i = 0; i < ln; i++) pa[i] = r1[i];
        for (int i = 0; i < lm; i++) pa[ln + i] = rho[i];
        for (int i = 0; i < lm; i++) pb[i] = rho[i];
        for (int i = 0; i < lk; i++) pb[lm + i] = r2[i];
        uint64_t ea, eb;
        mle_int(A, ln + lm, pa, &ea);
        mle_int(B, lm + lk, pb, &eb);
        free(pa);
        free(pb);
        if (ea != info->a_star || eb != info->b_star) { verdict = 3; goto done; }
    }
    /* 4: C = 2^s R + E with E = Rm - 2^(s-1), so C~(r) = 2^s R~(r) + Rm~(r) - 2^(s-1) */
    {
        uint64_t rhs = fadd(fmul(fpow2(s), info->r_claim), info->rm_claim);
        if (mode == 0) rhs = fsub(rhs, fpow2(s - 1));
        if (rhs != info->c0) { verdict = 4; goto done; }
    }
    /* 5-6: range sum-check chain and its final identity */
    {
        uint64_t H = fadd(fmul(lam[0], info->rm_claim), fmul(lam[1], fadd(info->r_claim, fpow2(t + 1))));
        if (relu) H = fadd(H, fmul(lam[2], info->y_claim));
        H = fmul(mu, H);
        if (!sumcheck_chain(lP + lN, 3, H, rs_evals, sigma, &fin)) { verdict = 5; goto done; }
        uint64_t W[128];
        plane_weights(W, P, s, t, relu, lam);
        uint64_t wsig, eqp = 1, eqx = 1;
        mle_field(W, lP, sigma, &wsig);
        for (int i = 0; i < lP; i++)
            eqp = fmul(eqp, fadd(fmul(tau_p[i], sigma[i]), fmul(fsub(1, tau_p[i]), fsub(1, sigma[i]))));
        for (int i = 0; i < lN; i++)
            eqx = fmul(eqx, fadd(fmul(r12[i], sigma[lP + i]), fmul(fsub(1, r12[i]), fsub(1, sigma[lP + i]))));
        uint64_t bc = info->bits_claim;
        uint64_t expect = fadd(fmul(fmul(eqp, eqx), fmul(bc, fsub(bc, 1))), fmul(mu, fmul(fmul(wsig, eqx), bc)));
        if (fin != expect) { verdict = 6; goto done; }
        /* 7: open the bit table at sigma */
        uint64_t eb;
        mle_int(bits, lP + lN, sigma, &eb);
        if (eb != bc) { verdict = 7; goto done; }
    }
    /* 8: open R, Rm, Y at (r1, r2) */
    {
        uint64_t er, erm, ey;
        mle_int(R, lN, r12, &er);
        mle_int(Rm, lN, r12, &erm);
        mle_int(Y, lN, r12, &ey);
        if (er != info->r_claim || erm != info->rm_claim || ey != info->y_claim) { verdict = 8; goto done; }
    }
    /* 9-10: ReLU zero-check chain from 0, final identity, openings at rho' */
    if (relu) {
        if (!sumcheck_chain(lN, 3, 0, zc_evals, rho2, &fin)) { verdict = 9; goto done; }
        uint64_t eqx = 1;
        for (int i = 0; i < lN; i++)
            eqx = fmul(eqx, fadd(fmul(r12[i], rho2[i]), fmul(fsub(1, r12[i]), fsub(1, rho2[i]))));
        uint64_t expect = fmul(eqx, fsub(fmul(info->r_at, info->r_at), fmul(info->y_at, info->y_at)));
        if (fin != expect) { verdict = 9; goto done; }
        uint64_t er, ey;
        mle_int(R, lN, rho2, &er);
        mle_int(Y, lN, rho2, &ey);
        if (er != info->r_at || ey != info->y_at) { verdict = 10; goto done; }
    }
    /* 11: 2 Z = R + Y (Sec. IV, ReLU verification) or Z = R, and Z opening */
    {
        uint64_t ez;
        if (relu) {
            if (fmul(2, info->z_claim) != fadd(info->r_claim, info->y_claim)) { verdict = 11; goto done; }
        } else if (info->z_claim != info->r_claim) { verdict = 11; goto done; }
        mle_int(Z, lN, r12, &ez);
        if (ez != info->z_claim) { verdict = 11; goto done; }
    }
    (void)N;
done:
    free(r12);
    return verdict;
}

/* ------------------------------------------------------------------------ */
/* Layer composition through a gather (Sec. III-C chains layers; the paper  */
/* is silent on convolutions, whose inputs are gathers of the previous      */
/* layer's output: im2col, flattening).                                     */
/* ------------------------------------------------------------------------ */

/*
 * The next layer's input is A[a] = Z[src[a]] for src[a] >= 0 and 0 for
 * src[a] < 0 (a = row * m + col, na = n * m entries, Z of nz entries).  Its
 * multilinear extension at a point z of log na variables is
 *     A~(z) = sum_a eq(z, a) A[a] = sum_y Z[y] W_z[y],
 *     W_z[y] = sum over the a with src[a] = y of eq(z, a),
 * a sum over y of the product of two multilinear tables, so a degree-2
 * sum-check (Sec. II-D) over log nz variables reduces the claim A~(z) to
 * Z~(y*) W~_z(y*) at the point y* of its challenges.  Z~(y*) is a claim on
 * the previous layer's output; W~_z(y*) = sum_a eq(z, a) eq(y*, src[a]) is
 * computable from the public gather map.
 *
 * Consumes log nz challenges at *cursor.  evals: 3 log nz words (g_j(0..2)).
 */
int orc_link_prove(int64_t na, const int64_t *src, const uint64_t *z, int64_t nz, const int64_t *Z,
                   const uint64_t *chal, int64_t nchal, int64_t *cursor, uint64_t *evals, uint64_t *claim,
                   uint64_t *z_at, uint64_t *w_at)
{
    int va = ilog2_exact(na), vz = ilog2_exact(nz);
    if (va < 0 || vz < 0) return ORC_E_INVAL;
    if (*cursor < 0 || *cursor + vz > nchal) return ORC_E_CHALLENGES;
    for (int64_t a = 0; a < na; a++)
        if (src[a] >= nz) return ORC_E_INVAL;
    uint64_t *eqz = malloc(sizeof(uint64_t) * (size_t)na);
    uint64_t *W = calloc((size_t)nz, sizeof(uint64_t));
    uint64_t *T = malloc(sizeof(uint64_t) * (size_t)nz);
    if (!eqz || !W || !T) {
        free(eqz);
        free(W);
        free(T);
        return ORC_E_NOMEM;
    }
    chi_vector(z, va, eqz);
    for (int64_t a = 0; a < na; a++)
        if (src[a] >= 0) W[src[a]] = fadd(W[src[a]], eqz[a]);
    uint64_t c = 0;
    for (int64_t y = 0; y < nz; y++) {
        T[y] = fint(Z[y]);
        c = fadd(c, fmul(T[y], W[y]));
    }
    *claim = c;
    uint64_t *tabs[2] = {T, W}, finals[2];
    sumcheck_prove(vz, 2, 2, tabs, summand_matmul, NULL, chal + *cursor, evals, finals);
    *z_at = finals[0];
    *w_at = finals[1];
    *cursor += vz;
    free(eqz);
    free(W);
    free(T);
    return ORC_OK;
}

/*
 * Verifier of a gather link: 0 accept, 15 reject.  a_star is the claim
 * A~(z) the next layer's matrix sum-check ended with; Z is the previous
 * layer's (opened) output.  Checks the chain from a_star, the final product
 * z_at w_at, z_at against Z~(y*) and w_at against sum_a eq(z, a) eq(y*, src[a]).
 */
int orc_link_verify(int64_t na, const int64_t *src, const uint64_t *z, int64_t nz, const int64_t *Z,
                    uint64_t a_star, const uint64_t *evals, uint64_t claim, uint64_t z_at, uint64_t w_at,
                    const uint64_t *chal, int64_t nchal, int64_t *cursor)
{
    int va = ilog2_exact(na), vz = ilog2_exact(nz);
    if (va < 0 || vz < 0) return 15;
    if (*cursor < 0 || *cursor + vz > nchal) return 15;
    const uint64_t *ys = chal + *cursor;
    *cursor += vz;
    if (claim != a_star || z_at >= ORC_P || w_at >= ORC_P) return 15;
    uint64_t fin;
    if (!sumcheck_chain(vz, 2, claim, evals, ys, &fin)) return 15;
    if (fin != fmul(z_at, w_at)) return 15;
    uint64_t ez;
    if (mle_int(Z, vz, ys, &ez) != 0 || ez != z_at) return 15;
    uint64_t *ea = malloc(sizeof(uint64_t) * (size_t)na), *ey = malloc(sizeof(uint64_t) * (size_t)nz);
    if (!ea || !ey) {
        free(ea);
        free(ey);
        return ORC_E_NOMEM;
    }
    chi_vector(z, va, ea);
    chi_vector(ys, vz, ey);
    uint64_t w = 0;
    int bad = 0;
    for (int64_t a = 0; a < na && !bad; a++) {
        if (src[a] < 0) continue;
        if (src[a] >= nz) bad = 1;
        else w = fadd(w, fmul(ea[a], ey[src[a]]));
    }
    free(ea);
    free(ey);
    return !bad && w == w_at ? 0 : 15;
}
