// verify.cpp -- host-only verifier of the C ABI (ra_verify), Sec. IV.
//
// The verifier replays the challenge stream and checks, per layer: the three
// sum-check chains (Sec. II-D: g_j(0) + g_j(1) equals the previous round's
// polynomial at its challenge), each instance's final identity, the rounding
// link between the matrix claim and the rounded output (Theorem A.1,
// condition 1), the ReLU output link 2 Z = R + Y (Sec. IV), the field guard,
// and opens the tables handed over in place of commitments by evaluating
// their multilinear extensions (Eq. (1)) at the challenge points.
#include <algorithm>
#include <cstring>
#include <functional>
#include <vector>

#include "ra.h"
#include "secp256k1.hpp"
#include "sha256.hpp"
#include "stream.hpp"

namespace {

constexpr uint64_t kP = 0x1FFFFFFFFFFFFFFFull;
typedef unsigned __int128 u128;

// host arithmetic modulo 2^61 - 1 by folding at bit 61
uint64_t fold(u128 x)
{
    uint64_t lo = (uint64_t)x & kP;
    u128 rest = x >> 61;
    while (rest) {
        x = (u128)lo + rest;
        lo = (uint64_t)x & kP;
        rest = x >> 61;
    }
    return lo == kP ? 0 : lo;
}
uint64_t fadd(uint64_t a, uint64_t b) { return fold((u128)a + b); }
uint64_t fsub(uint64_t a, uint64_t b) { return fold((u128)a + kP - b); }
uint64_t fmul(uint64_t a, uint64_t b) { return fold((u128)a * b); }
uint64_t fint(int64_t z) { return z >= 0 ? fold((u128)(uint64_t)z) : fsub(0, fold((u128)(uint64_t)(-(z + 1)) + 1)); }
uint64_t fpow(uint64_t b, uint64_t e)
{
    uint64_t r = 1;
    while (e) {
        if (e & 1) r = fmul(r, b);
        b = fmul(b, b);
        e >>= 1;
    }
    return r;
}
uint64_t eq1(uint64_t a, uint64_t b) { return fadd(fmul(a, b), fmul(fsub(1, a), fsub(1, b))); }

bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }
int log2u(uint64_t x)
{
    int l = 0;
    while ((1ull << l) < x) l++;
    return l;
}

// value at x of the polynomial of degree d through (i, e[i]), i = 0..d
uint64_t lagrange(const uint64_t *e, int d, uint64_t x)
{
    uint64_t acc = 0;
    for (int i = 0; i <= d; i++) {
        uint64_t num = 1, den = 1;
        for (int j = 0; j <= d; j++) {
            if (j == i) continue;
            num = fmul(num, fsub(x, (uint64_t)j));
            den = fmul(den, fint(i - j));
        }
        acc = fadd(acc, fmul(e[i], fmul(num, fpow(den, kP - 2))));
    }
    return acc;
}

// Checks one sum-check transcript; returns false on a broken chain.
bool chain(int rounds, int d, uint64_t claim, const uint64_t *evals, const uint64_t *rho, uint64_t *final_value)
{
    uint64_t cur = claim;
    for (int j = 0; j < rounds; j++) {
        const uint64_t *g = evals + (size_t)j * (d + 1);
        if (fadd(g[0], g[1]) != cur) return false;
        cur = lagrange(g, d, rho[j]);
    }
    *final_value = cur;
    return true;
}

// Multilinear extension of a table at z by binding its variables one at a
// time, most significant first: T[i] <- T[i] + z_j (T[i + h] - T[i]).
uint64_t mle_bind_all(std::vector<uint64_t> T, const uint64_t *z, int v)
{
    size_t size = T.size();
    for (int j = 0; j < v; j++) {
        const size_t h = size / 2;
        for (size_t i = 0; i < h; i++) T[i] = fadd(T[i], fmul(z[j], fsub(T[i + h], T[i])));
        size = h;
    }
    return T[0];
}

template <typename I> uint64_t mle_ints(const I *tab, size_t len, const uint64_t *z, int v)
{
    std::vector<uint64_t> T(len);
    for (size_t i = 0; i < len; i++) T[i] = fint((int64_t)tab[i]);
    return mle_bind_all(std::move(T), z, v);
}

// The 2^v values eq(z, y), y's most significant bit paired with z_0 (the
// order in which mle_bind_all binds): each variable doubles the table.
std::vector<uint64_t> eq_table(const uint64_t *z, int v)
{
    std::vector<uint64_t> T(1, 1);
    for (int i = 0; i < v; i++) {
        std::vector<uint64_t> U(T.size() * 2);
        for (size_t y = 0; y < T.size(); y++) {
            U[2 * y + 1] = fmul(T[y], z[i]);
            U[2 * y] = fsub(T[y], U[2 * y + 1]);
        }
        T.swap(U);
    }
    return T;
}

uint64_t eq_points(const uint64_t *a, const uint64_t *b, int v)
{
    uint64_t acc = 1;
    for (int i = 0; i < v; i++) acc = fmul(acc, eq1(a[i], b[i]));
    return acc;
}

int verify_layer(const ra_layer_public &L, const ra_layer_tables &T, const ra_layer_transcript &tr,
                 const ra_layer_public *prev, const uint64_t *chal, uint64_t nchal, uint64_t *cursor,
                 ra_status *err)
{
    const uint32_t n = L.n, m = L.m, k = L.k;
    if (!is_pow2(n) || !is_pow2(m) || !is_pow2(k) || (!L.A && !L.link_src) || !L.B || !L.Z || !T.R || !T.Rm ||
        !T.Y || !T.bits)
        return 13;
    if ((L.a_dtype != RA_I16 && L.a_dtype != RA_I32) || L.s < 1 || L.s > 30 || L.relu > 1 || L.round_mode > 1)
        return 13;
    if (L.link_src && L.chained) return 13;
    const int ln = log2u(n), lm = log2u(m), lk = log2u(k), lN = ln + lk;
    const uint64_t N = (uint64_t)n * k;
    const int s = (int)L.s, relu = (int)L.relu, t = tr.wit.t;
    // 14: chaining
    if (L.chained) {
        if (!prev || L.a_dtype != RA_I32 || prev->n != n || prev->k != m) return 14;
        const int32_t *A = (const int32_t *)L.A;
        for (uint64_t i = 0; i < (uint64_t)n * m; i++)
            if (A[i] != prev->Z[i]) return 14;
    }
    // 12: parameters
    if (t < 0 || s + t + 3 > 61 || tr.wit.s != L.s || tr.wit.relu != L.relu || tr.wit.round_mode != L.round_mode)
        return 12;
    const int Q = s + (t + 2) * (relu ? 2 : 1);
    int P = 1, lP = 0;
    while (P < Q) {
        P <<= 1;
        lP++;
    }
    if ((int)tr.wit.P != P || lP > 6) return 12;
    if (tr.mm.log_m != (uint32_t)lm || tr.rng.rounds != (uint32_t)(lP + lN) ||
        tr.rng.relu_rounds != (uint32_t)(relu ? lN : 0))
        return 13;
    if ((lm && !tr.mm.evals) || !tr.rng.evals || (relu && lN && !tr.rng.relu_evals)) return 13;
    std::vector<uint64_t> words = {tr.mm.c0, tr.mm.a_star, tr.mm.b_star, tr.wit.r_claim, tr.wit.rm_claim,
                                   tr.wit.y_claim, tr.wit.z_claim, tr.rng.range_sum, tr.rng.bits_claim,
                                   tr.rng.r_at, tr.rng.y_at};
    for (int i = 0; i < 3 * lm; i++) words.push_back(tr.mm.evals[i]);
    for (int i = 0; i < 4 * (lP + lN); i++) words.push_back(tr.rng.evals[i]);
    if (relu)
        for (int i = 0; i < 4 * lN; i++) words.push_back(tr.rng.relu_evals[i]);
    for (uint64_t w : words)
        if (w >= kP) return 12;

    const uint64_t need = (uint64_t)ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    if (*cursor + need > nchal) {
        *err = RA_E_SEED;
        return 13;
    }
    const uint64_t *r1 = chal + *cursor, *r2 = r1 + ln, *rho = r2 + lk, *lam = rho + lm;
    const uint64_t mu = lam[3], *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    *cursor += need;
    std::vector<uint64_t> r12(r1, r1 + ln);
    r12.insert(r12.end(), r2, r2 + lk);

    // 1-2: matrix-multiplication sum-check (Eq. (4))
    uint64_t fin;
    if (!chain(lm, 2, tr.mm.c0, tr.mm.evals, rho, &fin)) return 1;
    if (fin != fmul(tr.mm.a_star, tr.mm.b_star)) return 2;
    // 3: a* = A~(r1, rho) (with a gather link: checked by the link, 15), b* = B~(rho, r2)
    std::vector<uint64_t> pa(r1, r1 + ln);
    pa.insert(pa.end(), rho, rho + lm);
    {
        std::vector<uint64_t> pb(rho, rho + lm);
        pb.insert(pb.end(), r2, r2 + lk);
        if (!L.link_src) {
            const uint64_t ea = L.a_dtype == RA_I16
                                    ? mle_ints((const int16_t *)L.A, (size_t)n * m, pa.data(), ln + lm)
                                    : mle_ints((const int32_t *)L.A, (size_t)n * m, pa.data(), ln + lm);
            if (ea != tr.mm.a_star) return 3;
        }
        const uint64_t eb = mle_ints(L.B, (size_t)m * k, pb.data(), lm + lk);
        if (eb != tr.mm.b_star) return 3;
    }
    // 4: C = 2^s R + Rm - 2^(s-1) (floor mode: C = 2^s R + Rm), at (r1, r2)
    {
        uint64_t rhs = fadd(fmul(fint((int64_t)1 << s), tr.wit.r_claim), tr.wit.rm_claim);
        if (L.round_mode == RA_ROUND_NEAREST) rhs = fsub(rhs, fint((int64_t)1 << (s - 1)));
        if (rhs != tr.mm.c0) return 4;
    }
    // 5-7: concatenated range sum-check
    {
        uint64_t H = fadd(fmul(lam[0], tr.wit.rm_claim), fmul(lam[1], fadd(tr.wit.r_claim, fint((int64_t)1 << (t + 1)))));
        if (relu) H = fadd(H, fmul(lam[2], tr.wit.y_claim));
        H = fmul(mu, H);
        if (H != tr.rng.range_sum) return 5;
        if (!chain(lP + lN, 3, H, tr.rng.evals, sigma, &fin)) return 5;
        std::vector<uint64_t> W(P, 0);
        int q = 0;
        for (int b = 0; b < s; b++) W[q++] = fmul(lam[0], 1ull << b);
        for (int b = 0; b < t + 2; b++) W[q++] = fmul(lam[1], 1ull << b);
        if (relu)
            for (int b = 0; b < t + 2; b++) W[q++] = fmul(lam[2], 1ull << b);
        const uint64_t wsig = mle_bind_all(W, sigma, lP);
        const uint64_t ep = eq_points(tau_p, sigma, lP), ex = eq_points(r12.data(), sigma + lP, lN);
        const uint64_t bc = tr.rng.bits_claim;
        const uint64_t want = fadd(fmul(fmul(ep, ex), fmul(bc, fsub(bc, 1))), fmul(mu, fmul(fmul(wsig, ex), bc)));
        if (fin != want) return 6;
        // 7: b~(sigma): bind the plane variables word by word, then the x variables
        std::vector<uint64_t> eqp(P);
        for (int qq = 0; qq < P; qq++) {
            uint64_t acc = 1;
            for (int i = 0; i < lP; i++) acc = fmul(acc, eq1(sigma[i], (uint64_t)((qq >> (lP - 1 - i)) & 1)));
            eqp[qq] = acc;
        }
        std::vector<uint64_t> bx(N);
        for (uint64_t x = 0; x < N; x++) {
            const uint64_t w = T.bits[x];
            if (P < 64 && (w >> P)) return 7;  // bits beyond the plane count
            uint64_t acc = 0;
            for (int qq = 0; qq < P; qq++)
                if ((w >> qq) & 1) acc = fadd(acc, eqp[qq]);
            bx[x] = acc;
        }
        if (mle_bind_all(std::move(bx), sigma + lP, lN) != bc) return 7;
    }
    // 8: openings of R, Rm, Y at (r1, r2)
    if (mle_ints(T.R, N, r12.data(), lN) != tr.wit.r_claim || mle_ints(T.Rm, N, r12.data(), lN) != tr.wit.rm_claim ||
        mle_ints(T.Y, N, r12.data(), lN) != tr.wit.y_claim)
        return 8;
    // 9-10: ReLU zero-check (Eq. (6)) from 0, its final identity, openings at rho'
    if (relu) {
        if (!chain(lN, 3, 0, tr.rng.relu_evals, rho2, &fin)) return 9;
        const uint64_t ex = eq_points(r12.data(), rho2, lN);
        if (fin != fmul(ex, fsub(fmul(tr.rng.r_at, tr.rng.r_at), fmul(tr.rng.y_at, tr.rng.y_at)))) return 9;
        if (mle_ints(T.R, N, rho2, lN) != tr.rng.r_at || mle_ints(T.Y, N, rho2, lN) != tr.rng.y_at) return 10;
    }
    // 11: output link and the public output's opening
    if (relu) {
        if (fmul(2, tr.wit.z_claim) != fadd(tr.wit.r_claim, tr.wit.y_claim)) return 11;
    } else if (tr.wit.z_claim != tr.wit.r_claim) {
        return 11;
    }
    if (mle_ints(L.Z, N, r12.data(), lN) != tr.wit.z_claim) return 11;
    // 15: the gather link A[a] = Z_prev[src[a]]: a* = sum_y Z_prev[y] W[y]
    // reduced by a degree-2 sum-check to Z_prev~(y*) W~(y*)
    if (L.link_src) {
        if (!prev || !prev->Z) return 15;
        const uint64_t nz = (uint64_t)prev->n * prev->k;
        const int vz = log2u(nz);
        const ra_link_proof &lnk = tr.link;
        if (lnk.rounds != (uint32_t)vz || (vz && !lnk.evals)) return 15;
        if (*cursor + vz > nchal) {
            *err = RA_E_SEED;
            return 15;
        }
        const uint64_t *ys = chal + *cursor;
        *cursor += vz;
        if (lnk.claim != tr.mm.a_star || lnk.z_at >= kP || lnk.w_at >= kP) return 15;
        for (int i = 0; i < 3 * vz; i++)
            if (lnk.evals[i] >= kP) return 15;
        if (!chain(vz, 2, lnk.claim, lnk.evals, ys, &fin)) return 15;
        if (fin != fmul(lnk.z_at, lnk.w_at)) return 15;
        if (mle_ints(prev->Z, nz, ys, vz) != lnk.z_at) return 15;
        const std::vector<uint64_t> ea = eq_table(pa.data(), ln + lm), ey = eq_table(ys, vz);
        uint64_t w = 0;
        for (uint64_t a = 0; a < (uint64_t)n * m; a++) {
            const int32_t y = L.link_src[a];
            if (y == -1) continue;
            if (y < 0 || (uint64_t)y >= nz) return 15;
            w = fadd(w, fmul(ea[a], ey[y]));
        }
        if (w != lnk.w_at) return 15;
    }
    return 0;
}

}  // namespace

extern "C" ra_status ra_verify_stream(uint64_t p, const uint64_t *h_challenges, uint64_t n_challenges,
                                      uint32_t n_layers, const ra_layer_public *pub, const ra_layer_tables *tables,
                                      const ra_layer_transcript *tr, int32_t *verdict, uint32_t *failed_layer)
{
    if (!verdict || !failed_layer || (n_layers && (!pub || !tables || !tr)) || (n_challenges && !h_challenges))
        return RA_E_INVAL;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    for (uint64_t i = 0; i < n_challenges; i++)
        if (h_challenges[i] >= kP) return RA_E_SEED;
    *verdict = 0;
    *failed_layer = 0;
    uint64_t cursor = 0;
    for (uint32_t l = 0; l < n_layers; l++) {
        ra_status err = RA_OK;
        const int v = verify_layer(pub[l], tables[l], tr[l], l ? &pub[l - 1] : nullptr, h_challenges, n_challenges,
                                   &cursor, &err);
        if (err != RA_OK) return err;
        if (v) {
            *verdict = v;
            *failed_layer = l;
            return RA_OK;
        }
    }
    return RA_OK;
}

// The seeded form draws as many challenges as the layers consume (their
// dimensions and plane counts as stated; a malformed layer fails its own
// checks before it reads any) and verifies against them.
extern "C" ra_status ra_verify(uint64_t p, uint64_t seed, uint32_t n_layers, const ra_layer_public *pub,
                               const ra_layer_tables *tables, const ra_layer_transcript *tr, int32_t *verdict,
                               uint32_t *failed_layer)
{
    if (!verdict || !failed_layer || (n_layers && (!pub || !tables || !tr))) return RA_E_INVAL;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    if (seed == 0) return RA_E_SEED;
    uint64_t total = 0;
    auto lg = [](uint64_t x) { return is_pow2(x) && x <= (1ull << 32) ? log2u(x) : 0; };
    for (uint32_t l = 0; l < n_layers; l++) {
        const int ln = lg(pub[l].n), lm = lg(pub[l].m), lk = lg(pub[l].k), lN = ln + lk;
        const int lP = is_pow2(tr[l].wit.P) && tr[l].wit.P <= 128 ? log2u(tr[l].wit.P) : 0;
        total += (uint64_t)ln + lk + lm + 4 + 2 * lP + lN + (pub[l].relu ? lN : 0);
        if (pub[l].link_src && l > 0) total += (uint64_t)lg(pub[l - 1].n) + lg(pub[l - 1].k);
    }
    std::vector<uint64_t> chal(total ? total : 1);
    ra::ChallengeStream cs(seed);
    for (uint64_t i = 0; i < total; i++) chal[i] = cs.next();
    return ra_verify_stream(p, chal.data(), total, n_layers, pub, tables, tr, verdict, failed_layer);
}

// ---------------------------------------------------------------------------
// The verifier for layers proven with challenges in F_{p^2} = F_p[i] /
// (i^2 + 1): the checks of verify_layer, same numbering, every transcript
// element a pair (re, im).
// ---------------------------------------------------------------------------
namespace {

struct G2 {
    uint64_t re, im;
};
G2 g2(uint64_t a) { return G2{a, 0}; }
G2 g2add(G2 a, G2 b) { return G2{fadd(a.re, b.re), fadd(a.im, b.im)}; }
G2 g2sub(G2 a, G2 b) { return G2{fsub(a.re, b.re), fsub(a.im, b.im)}; }
G2 g2mul(G2 a, G2 b)
{
    return G2{fsub(fmul(a.re, b.re), fmul(a.im, b.im)), fadd(fmul(a.re, b.im), fmul(a.im, b.re))};
}
G2 g2scale(G2 a, uint64_t c) { return G2{fmul(a.re, c), fmul(a.im, c)}; }
bool g2same(G2 a, G2 b) { return a.re == b.re && a.im == b.im; }
G2 g2of(const ra_fp2 &v) { return G2{v.re, v.im}; }
G2 g2eq1(G2 a, G2 b) { return g2add(g2mul(a, b), g2mul(g2sub(g2(1), a), g2sub(g2(1), b))); }

G2 lagrange2(const G2 *e, int d, G2 x)
{
    G2 acc = g2(0);
    for (int i = 0; i <= d; i++) {
        G2 num = g2(1);
        uint64_t den = 1;
        for (int j = 0; j <= d; j++) {
            if (j == i) continue;
            num = g2mul(num, g2sub(x, g2((uint64_t)j)));
            den = fmul(den, fint(i - j));
        }
        acc = g2add(acc, g2mul(e[i], g2scale(num, fpow(den, kP - 2))));
    }
    return acc;
}

bool chain2(int rounds, int d, G2 claim, const ra_fp2 *evals, const G2 *rho, G2 *final_value)
{
    G2 cur = claim;
    std::vector<G2> g(d + 1);
    for (int j = 0; j < rounds; j++) {
        for (int X = 0; X <= d; X++) g[X] = g2of(evals[(size_t)j * (d + 1) + X]);
        if (!g2same(g2add(g[0], g[1]), cur)) return false;
        cur = lagrange2(g.data(), d, rho[j]);
    }
    *final_value = cur;
    return true;
}

G2 bind_all2(std::vector<G2> T, const G2 *z, int v)
{
    size_t size = T.size();
    for (int j = 0; j < v; j++) {
        const size_t h = size / 2;
        for (size_t i = 0; i < h; i++) T[i] = g2add(T[i], g2mul(z[j], g2sub(T[i + h], T[i])));
        size = h;
    }
    return T[0];
}

template <typename I> G2 mle_ints2(const I *tab, size_t len, const G2 *z, int v)
{
    std::vector<G2> T(len);
    for (size_t i = 0; i < len; i++) T[i] = g2(fint((int64_t)tab[i]));
    return bind_all2(std::move(T), z, v);
}

G2 eq_points2(const G2 *a, const G2 *b, int v)
{
    G2 acc = g2(1);
    for (int i = 0; i < v; i++) acc = g2mul(acc, g2eq1(a[i], b[i]));
    return acc;
}

// The sizes a layer's challenge source needs (verify_layer_fp2).
struct LayerShape {
    int ln, lk, lm, lP, lN, t, P, relu;
};
// Fills c with the layer's challenges in protocol order; false: unavailable.
using DrawFn = std::function<bool(const LayerShape &, std::vector<G2> &)>;

int verify_layer_fp2(const ra_layer_public &L, const ra_layer_tables &T, const ra_layer_proof_fp2 &tr,
                     const ra_layer_public *prev, const DrawFn &draw)
{
    const uint32_t n = L.n, m = L.m, k = L.k;
    if (!is_pow2(n) || !is_pow2(m) || !is_pow2(k) || !L.A || !L.B || !L.Z || !T.R || !T.Rm || !T.Y || !T.bits)
        return 13;
    if ((L.a_dtype != RA_I16 && L.a_dtype != RA_I32) || L.s < 1 || L.s > 30 || L.relu > 1 || L.round_mode > 1)
        return 13;
    const int ln = log2u(n), lm = log2u(m), lk = log2u(k), lN = ln + lk;
    const uint64_t N = (uint64_t)n * k;
    const int s = (int)L.s, relu = (int)L.relu, t = tr.t;
    if (L.link_src) return 13;  // gather links are proven over F_p only
    if (L.chained) {
        if (!prev || L.a_dtype != RA_I32 || prev->n != n || prev->k != m) return 14;
        const int32_t *A = (const int32_t *)L.A;
        for (uint64_t i = 0; i < (uint64_t)n * m; i++)
            if (A[i] != prev->Z[i]) return 14;
    }
    if (t < 0 || s + t + 3 > 61 || tr.s != L.s || tr.relu != L.relu || tr.round_mode != L.round_mode) return 12;
    const int Q = s + (t + 2) * (relu ? 2 : 1);
    int P = 1, lP = 0;
    while (P < Q) {
        P <<= 1;
        lP++;
    }
    if ((int)tr.P != P || lP > 6) return 12;
    if (tr.log_m != (uint32_t)lm || tr.rounds != (uint32_t)(lP + lN) || tr.relu_rounds != (uint32_t)(relu ? lN : 0))
        return 13;
    if ((lm && !tr.mm_evals) || !tr.rs_evals || (relu && lN && !tr.zc_evals)) return 13;
    std::vector<ra_fp2> words = {tr.c0, tr.a_star, tr.b_star, tr.r_claim, tr.rm_claim, tr.y_claim, tr.z_claim,
                                 tr.range_sum, tr.bits_claim, tr.r_at, tr.y_at};
    for (int i = 0; i < 3 * lm; i++) words.push_back(tr.mm_evals[i]);
    for (int i = 0; i < 4 * (lP + lN); i++) words.push_back(tr.rs_evals[i]);
    if (relu)
        for (int i = 0; i < 4 * lN; i++) words.push_back(tr.zc_evals[i]);
    for (const ra_fp2 &w : words)
        if (w.re >= kP || w.im >= kP) return 12;

    const uint64_t need = (uint64_t)ln + lk + lm + 4 + lP + (lP + lN) + (relu ? lN : 0);
    std::vector<G2> c(need);
    if (!draw(LayerShape{ln, lk, lm, lP, lN, t, P, relu}, c) || c.size() != need) return 13;
    const G2 *r1 = c.data(), *r2 = r1 + ln, *rho = r2 + lk, *lam = rho + lm;
    const G2 mu = lam[3], *tau_p = lam + 4, *sigma = tau_p + lP, *rho2 = sigma + lP + lN;
    std::vector<G2> r12(r1, r1 + ln);
    r12.insert(r12.end(), r2, r2 + lk);

    G2 fin;
    if (!chain2(lm, 2, g2of(tr.c0), tr.mm_evals, rho, &fin)) return 1;
    if (!g2same(fin, g2mul(g2of(tr.a_star), g2of(tr.b_star)))) return 2;
    {
        std::vector<G2> pa(r1, r1 + ln), pb(rho, rho + lm);
        pa.insert(pa.end(), rho, rho + lm);
        pb.insert(pb.end(), r2, r2 + lk);
        const G2 ea = L.a_dtype == RA_I16 ? mle_ints2((const int16_t *)L.A, (size_t)n * m, pa.data(), ln + lm)
                                          : mle_ints2((const int32_t *)L.A, (size_t)n * m, pa.data(), ln + lm);
        const G2 eb = mle_ints2(L.B, (size_t)m * k, pb.data(), lm + lk);
        if (!g2same(ea, g2of(tr.a_star)) || !g2same(eb, g2of(tr.b_star))) return 3;
    }
    {
        G2 rhs = g2add(g2scale(g2of(tr.r_claim), fint((int64_t)1 << s)), g2of(tr.rm_claim));
        if (L.round_mode == RA_ROUND_NEAREST) rhs = g2sub(rhs, g2(fint((int64_t)1 << (s - 1))));
        if (!g2same(rhs, g2of(tr.c0))) return 4;
    }
    {
        G2 H = g2add(g2mul(lam[0], g2of(tr.rm_claim)),
                     g2mul(lam[1], g2add(g2of(tr.r_claim), g2(fint((int64_t)1 << (t + 1))))));
        if (relu) H = g2add(H, g2mul(lam[2], g2of(tr.y_claim)));
        H = g2mul(mu, H);
        if (!g2same(H, g2of(tr.range_sum))) return 5;
        if (!chain2(lP + lN, 3, H, tr.rs_evals, sigma, &fin)) return 5;
        std::vector<G2> W(P, g2(0));
        int q = 0;
        for (int b = 0; b < s; b++) W[q++] = g2scale(lam[0], 1ull << b);
        for (int b = 0; b < t + 2; b++) W[q++] = g2scale(lam[1], 1ull << b);
        if (relu)
            for (int b = 0; b < t + 2; b++) W[q++] = g2scale(lam[2], 1ull << b);
        const G2 wsig = bind_all2(W, sigma, lP);
        const G2 ep = eq_points2(tau_p, sigma, lP), ex = eq_points2(r12.data(), sigma + lP, lN);
        const G2 bc = g2of(tr.bits_claim);
        const G2 want = g2add(g2mul(g2mul(ep, ex), g2mul(bc, g2sub(bc, g2(1)))), g2mul(mu, g2mul(g2mul(wsig, ex), bc)));
        if (!g2same(fin, want)) return 6;
        std::vector<G2> eqp(P);
        for (int qq = 0; qq < P; qq++) {
            G2 acc = g2(1);
            for (int i = 0; i < lP; i++)
                acc = g2mul(acc, ((qq >> (lP - 1 - i)) & 1) ? sigma[i] : g2sub(g2(1), sigma[i]));
            eqp[qq] = acc;
        }
        std::vector<G2> bx(N);
        for (uint64_t x = 0; x < N; x++) {
            const uint64_t w = T.bits[x];
            if (P < 64 && (w >> P)) return 7;
            G2 acc = g2(0);
            for (int qq = 0; qq < P; qq++)
                if ((w >> qq) & 1) acc = g2add(acc, eqp[qq]);
            bx[x] = acc;
        }
        if (!g2same(bind_all2(std::move(bx), sigma + lP, lN), bc)) return 7;
    }
    if (!g2same(mle_ints2(T.R, N, r12.data(), lN), g2of(tr.r_claim)) ||
        !g2same(mle_ints2(T.Rm, N, r12.data(), lN), g2of(tr.rm_claim)) ||
        !g2same(mle_ints2(T.Y, N, r12.data(), lN), g2of(tr.y_claim)))
        return 8;
    if (relu) {
        if (!chain2(lN, 3, g2(0), tr.zc_evals, rho2, &fin)) return 9;
        const G2 ex = eq_points2(r12.data(), rho2, lN), ra = g2of(tr.r_at), ya = g2of(tr.y_at);
        if (!g2same(fin, g2mul(ex, g2sub(g2mul(ra, ra), g2mul(ya, ya))))) return 9;
        if (!g2same(mle_ints2(T.R, N, rho2, lN), ra) || !g2same(mle_ints2(T.Y, N, rho2, lN), ya)) return 10;
    }
    if (relu) {
        if (!g2same(g2scale(g2of(tr.z_claim), 2), g2add(g2of(tr.r_claim), g2of(tr.y_claim)))) return 11;
    } else if (!g2same(g2of(tr.z_claim), g2of(tr.r_claim))) {
        return 11;
    }
    if (!g2same(mle_ints2(L.Z, N, r12.data(), lN), g2of(tr.z_claim))) return 11;
    return 0;
}

}  // namespace

extern "C" ra_status ra_verify_fp2(uint64_t p, uint64_t seed, uint32_t n_layers, const ra_layer_public *pub,
                                   const ra_layer_tables *tables, const ra_layer_proof_fp2 *tr, int32_t *verdict,
                                   uint32_t *failed_layer)
{
    if (!verdict || !failed_layer || (n_layers && (!pub || !tables || !tr))) return RA_E_INVAL;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    if (seed == 0) return RA_E_SEED;
    *verdict = 0;
    *failed_layer = 0;
    ra::ChallengeStream cs(seed);
    const DrawFn draw = [&cs](const LayerShape &, std::vector<G2> &c) {
        for (G2 &x : c) {
            x.re = cs.next();
            x.im = cs.next();
        }
        return true;
    };
    for (uint32_t l = 0; l < n_layers; l++) {
        const int v = verify_layer_fp2(pub[l], tables[l], tr[l], l ? &pub[l - 1] : nullptr, draw);
        if (v) {
            *verdict = v;
            *failed_layer = l;
            return RA_OK;
        }
    }
    return RA_OK;
}

// ---------------------------------------------------------------------------
// The non-interactive verifier (Fiat-Shamir over F_{p^2}): the challenges are
// recovered by replaying the prover's transcript (the layer header, the
// caller's public digest, the Merkle root of the opened tables, then every
// message in the prover's order), then checked as in ra_verify_fp2.
// ---------------------------------------------------------------------------
namespace {

// Merkle root of the witness tables: R (LE32), Rm (LE16), Y (LE32), Z (LE32),
// the bit words (LE64), each zero-padded to 1 KiB chunks; leaf H(0x00 ||
// chunk), nodes H(0x01 || 4 digests), root H(0x02 || LE64(leaves) || top).
void witness_root(const ra_layer_tables &T, const int32_t *Z, uint64_t N, uint8_t out[32])
{
    struct Tab {
        const uint8_t *p;
        uint64_t bytes;
    } tabs[5] = {{(const uint8_t *)T.R, 4 * N}, {(const uint8_t *)T.Rm, 2 * N}, {(const uint8_t *)T.Y, 4 * N},
                 {(const uint8_t *)Z, 4 * N}, {(const uint8_t *)T.bits, 8 * N}};
    std::vector<uint8_t> dig;
    for (const Tab &tb : tabs)  // the host is little-endian: the tables' bytes are their LE encodings
        for (uint64_t off = 0; off < tb.bytes; off += 1024) {
            sha::Hasher h;
            h.init();
            h.byte(0x00);
            const uint64_t take = std::min<uint64_t>(1024, tb.bytes - off);
            h.update(tb.p + off, take);
            for (uint64_t i = take; i < 1024; i++) h.byte(0);
            uint8_t d[32];
            h.final(d);
            dig.insert(dig.end(), d, d + 32);
        }
    const uint64_t leaves = dig.size() / 32;
    uint64_t count = leaves;
    while (count > 1) {
        const uint64_t next = (count + 3) / 4;
        std::vector<uint8_t> up(32 * next);
        for (uint64_t g = 0; g < next; g++) {
            sha::Hasher h;
            h.init();
            h.byte(0x01);
            for (uint64_t c = 0; c < 4; c++) {
                if (4 * g + c < count) h.update(dig.data() + 32 * (4 * g + c), 32);
                else for (int i = 0; i < 32; i++) h.byte(0);
            }
            h.final(up.data() + 32 * g);
        }
        dig.swap(up);
        count = next;
    }
    sha::Hasher h;
    h.init();
    h.byte(0x02);
    h.le(leaves, 8);
    h.update(dig.data(), 32);
    h.final(out);
}

bool absorb_f2(sha::Transcript &fs, const ra_fp2 *v, int count)
{
    for (int i = 0; i < count; i++) {
        const uint64_t w[2] = {v[i].re, v[i].im};
        if (!sha::fs_absorb_words(fs, w, 2)) return false;
    }
    return true;
}

G2 draw2(sha::Transcript &fs)
{
    uint64_t w[2];
    sha::fs_draw(fs, w);
    return G2{w[0], w[1]};
}

}  // namespace

extern "C" ra_status ra_verify_fs(uint64_t p, const uint8_t *domain, uint32_t n_layers, const ra_layer_public *pub,
                                  const ra_layer_tables *tables, const ra_layer_proof_fp2 *tr,
                                  const uint8_t *pub_digests, int32_t *verdict, uint32_t *failed_layer)
{
    if (!verdict || !failed_layer || !domain || (n_layers && (!pub || !tables || !tr || !pub_digests)))
        return RA_E_INVAL;
    if (p != kP) return RA_E_UNSUPPORTED_PRIME;
    *verdict = 0;
    *failed_layer = 0;
    sha::Transcript fs;
    sha::fs_init(fs, domain);
    for (uint32_t l = 0; l < n_layers; l++) {
        const ra_layer_public &L = pub[l];
        const ra_layer_tables &T = tables[l];
        const ra_layer_proof_fp2 &t = tr[l];
        const uint8_t *pd = pub_digests + 32 * (size_t)l;
        const DrawFn replay = [&](const LayerShape &sh, std::vector<G2> &c) {
            const uint64_t N = (uint64_t)L.n * L.k;
            uint8_t root[32];
            witness_root(T, L.Z, N, root);
            const uint32_t hdr[8] = {L.n, L.m, L.k, L.s, L.relu, L.round_mode, (uint32_t)sh.t, (uint32_t)sh.P};
            uint8_t hb[32];
            for (int i = 0; i < 8; i++)
                for (int j = 0; j < 4; j++) hb[4 * i + j] = (uint8_t)(hdr[i] >> (8 * j));
            if (!sha::fs_absorb(fs, hb, 32) || !sha::fs_absorb(fs, pd, 32) || !sha::fs_absorb(fs, root, 32))
                return false;
            size_t q = 0;
            for (int i = 0; i < sh.ln + sh.lk; i++) c[q++] = draw2(fs);
            for (int j = 0; j < sh.lm; j++) {
                if (!absorb_f2(fs, t.mm_evals + 3 * j, 3)) return false;
                c[q++] = draw2(fs);
            }
            const ra_fp2 sent[6] = {t.a_star, t.b_star, t.r_claim, t.rm_claim, t.y_claim, t.z_claim};
            if (!absorb_f2(fs, sent, 6)) return false;
            for (int i = 0; i < 4 + sh.lP; i++) c[q++] = draw2(fs);
            for (int j = 0; j < sh.lP + sh.lN; j++) {
                if (!absorb_f2(fs, t.rs_evals + 4 * j, 4)) return false;
                c[q++] = draw2(fs);
            }
            if (!absorb_f2(fs, &t.bits_claim, 1)) return false;
            if (sh.relu) {
                for (int j = 0; j < sh.lN; j++) {
                    if (!absorb_f2(fs, t.zc_evals + 4 * j, 4)) return false;
                    c[q++] = draw2(fs);
                }
                const ra_fp2 fin[2] = {t.r_at, t.y_at};
                if (!absorb_f2(fs, fin, 2)) return false;
            }
            return q == c.size();
        };
        const int v = verify_layer_fp2(L, T, t, l ? &pub[l - 1] : nullptr, replay);
        if (v) {
            *verdict = v;
            *failed_layer = l;
            return RA_OK;
        }
    }
    return RA_OK;
}

// ---------------------------------------------------------------------------
// Opening a commitment on the host: recompute sum_i v_i G_i (double-and-add
// per value) and compare the affine bytes.
// ---------------------------------------------------------------------------
extern "C" ra_status ra_commit_open(const void *h_values, ra_dtype dtype, uint64_t n, const void *h_gens,
                                    const uint8_t *commitment, int32_t *ok)
{
    if (!ok || !commitment || (n && (!h_values || !h_gens))) return RA_E_INVAL;
    if (dtype != RA_I16 && dtype != RA_U16 && dtype != RA_I32 && dtype != RA_U64) return RA_E_INVAL;
    const uint32_t *g = (const uint32_t *)h_gens;
    secp::Jac acc = secp::jac_inf();
    for (uint64_t i = 0; i < n; i++) {
        int64_t sv = 0;
        uint64_t mag = 0;
        bool neg = false;
        switch (dtype) {
        case RA_I16: sv = ((const int16_t *)h_values)[i]; break;
        case RA_I32: sv = ((const int32_t *)h_values)[i]; break;
        case RA_U16: mag = ((const uint16_t *)h_values)[i]; break;
        default: mag = ((const uint64_t *)h_values)[i]; break;
        }
        if (dtype == RA_I16 || dtype == RA_I32) {
            neg = sv < 0;
            mag = (uint64_t)(neg ? -sv : sv);
        }
        if (!mag) continue;
        secp::Aff G;
        for (int l = 0; l < 8; l++) {
            G.x.v[l] = g[16 * i + l];
            G.y.v[l] = g[16 * i + 8 + l];
        }
        secp::Jac term = secp::jac_inf();
        for (int b = 63; b >= 0; b--) {
            term = secp::jac_dbl(term);
            if ((mag >> b) & 1) term = secp::jac_add_aff(term, G);
        }
        acc = secp::jac_add(acc, neg ? secp::jac_neg(term) : term);
    }
    uint8_t got[64];
    secp::jac_encode(acc, got);
    *ok = std::memcmp(got, commitment, 64) == 0 ? 1 : 0;
    return RA_OK;
}
