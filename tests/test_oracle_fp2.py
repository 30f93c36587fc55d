"""Pins of the oracle's protocol over F_{p^2} = F_p[i] / (i^2 + 1)
(oracle/ra_oracle_fp2.c), each against something other than the oracle
itself: the field against the regular (2 x 2 matrix) representation and the
Frobenius map; the protocol against the F_p oracle (already pinned) on
challenges of F_p, against brute-force hypercube sums over F_{p^2}, and by
its verifier's accept / reject behaviour (Sec. IV)."""
import random

import numpy as np
import pytest

import brute
from brute_fp2 import Fp2, mle2, eq_point2, round_polys2
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

P = (1 << 61) - 1


def rnd2(rng):
    return (rng.randrange(P), rng.randrange(P))


def test_field_fp2():
    rng = random.Random(5)
    i = (0, 1)
    assert orc.f2mul(i, i) == (P - 1, 0)                               # i^2 = -1
    for _ in range(200):
        a, b, c = rnd2(rng), rnd2(rng), rnd2(rng)
        assert orc.f2mul(a, b) == (Fp2(*a) * Fp2(*b)).pair            # regular representation
        assert orc.f2mul(a, b) == orc.f2mul(b, a)
        assert orc.f2mul(orc.f2mul(a, b), c) == orc.f2mul(a, orc.f2mul(b, c))
        assert orc.f2mul(a, orc.f2inv(a)) == (1, 0)
    # Frobenius: a^p is the conjugate (i^p = -i for p = 3 mod 4): a polynomial
    # identity of the field that a wrong product breaks
    a = rnd2(rng)
    r, base, e = (1, 0), a, P
    while e:
        if e & 1:
            r = orc.f2mul(r, base)
        base = orc.f2mul(base, base)
        e >>= 1
    assert r == (a[0], (P - a[1]) % P)


def test_mle_fp2_brute():
    rng = random.Random(6)
    for v in (0, 1, 3):
        tab = [rng.randrange(-1000, 1000) for _ in range(1 << v)]
        z = [rnd2(rng) for _ in range(v)]
        assert orc.mle_int_fp2(tab, z) == mle2(tab, [Fp2(*p) for p in z]).pair


def real_stream(seed, count):
    """A stream whose F_{p^2} challenges all lie in F_p (odd words zero)."""
    base = inputs.xorshift64_stream(seed, count)
    out = np.zeros(2 * count, dtype=np.uint64)
    out[0::2] = base
    return base, out


@pytest.mark.parametrize("relu,mode", [(True, 0), (False, 1), (True, 1)])
def test_fp2_on_real_challenges_equals_fp(relu, mode):
    """F_p is a subfield: with every challenge in F_p the F_{p^2} transcript
    is the F_p oracle's, with zero imaginary parts."""
    rng = np.random.default_rng(31 + mode + 2 * relu)
    A = rng.integers(-700, 700, size=(8, 16))
    B = rng.integers(-700, 700, size=(16, 4))
    base, wide = real_stream(99 + mode, 400)
    o = orc.prove_layer(A, B, 6, relu, mode, base)
    o2 = orc.prove_layer_fp2(A, B, 6, relu, mode, wide)
    assert o2["cursor"] == 2 * o["cursor"] and o2["t"] == o["t"] and o2["P"] == o["P"]
    for key in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim", "range_sum",
                "bits_claim", "r_at", "y_at"):
        assert o2[key] == (o[key], 0), key
    for key in ("mm_evals", "rs_evals", "zc_evals"):
        assert o2[key] == [(v, 0) for v in o[key]], key
    for key in ("C", "R", "Rm", "Y", "Z", "bits"):
        assert np.array_equal(o2[key], o[key]), key


def test_fp2_round_polys_brute():
    """Every round polynomial of the three instances against direct sums over
    the hypercube of the extended summand, evaluated by Eq. (1) in F_{p^2}."""
    rng = np.random.default_rng(8)
    A = rng.integers(-60, 60, size=(2, 4))
    B = rng.integers(-60, 60, size=(4, 2))
    s, relu = 3, True
    chal = inputs.xorshift64_stream(1234, 400)
    o = orc.prove_layer_fp2(A, B, s, relu, 0, chal)
    n, m, k = 2, 4, 2
    ln, lm, lk = 1, 2, 1
    lP = o["P"].bit_length() - 1
    lN = ln + lk
    c = [Fp2(int(chal[2 * j]), int(chal[2 * j + 1])) for j in range(o["cursor"] // 2)]
    r1, r2 = c[:ln], c[ln:ln + lk]
    rho = c[ln + lk:ln + lk + lm]
    lam = c[ln + lk + lm:ln + lk + lm + 4]
    tau_p = c[ln + lk + lm + 4:ln + lk + lm + 4 + lP]
    sigma = c[ln + lk + lm + 4 + lP:ln + lk + lm + 4 + 2 * lP + lN]
    rho2 = c[ln + lk + lm + 4 + 2 * lP + lN:]
    Af, Bf = A.reshape(-1).tolist(), B.reshape(-1).tolist()
    # matrix instance: gamma(l) = A~(r1, l) B~(l, r2)
    g = round_polys2(lm, 2, lambda pt: mle2(Af, r1 + pt) * mle2(Bf, pt + r2), rho)
    assert [x for r in g for x in r] == o["mm_evals"]
    assert o["c0"] == (Fp2(*g[0][0]) + Fp2(*g[0][1])).pair          # g_1(0) + g_1(1) = C~(r1, r2)
    # range instance over b(q, x): eq(tau, .) b (b - 1) + mu W(q) eq(r12, x) b
    t = o["t"]
    W = [Fp2(0)] * o["P"]
    q = 0
    for b in range(s):
        W[q] = lam[0] * (1 << b); q += 1
    for b in range(t + 2):
        W[q] = lam[1] * (1 << b); q += 1
    for b in range(t + 2):
        W[q] = lam[2] * (1 << b); q += 1
    bits = o["bits"].reshape(-1).tolist()
    tau = tau_p + r1 + r2
    r12 = r1 + r2

    def f_range(pt):
        bb = mle2(bits, pt)
        return eq_point2(tau, pt) * bb * (bb - 1) + lam[3] * mle2(W, pt[:lP]) * eq_point2(r12, pt[lP:]) * bb

    g = round_polys2(lP + lN, 3, f_range, sigma)
    assert [x for r in g for x in r] == o["rs_evals"]
    Rl, Yl = o["R"].reshape(-1).tolist(), o["Y"].reshape(-1).tolist()

    def f_relu(pt):
        rr, yy = mle2(Rl, pt), mle2(Yl, pt)
        return eq_point2(r12, pt) * (rr * rr - yy * yy)

    g = round_polys2(lN, 3, f_relu, rho2)
    assert [x for r in g for x in r] == o["zc_evals"]
    assert o["r_at"] == mle2(Rl, rho2).pair and o["y_at"] == mle2(Yl, rho2).pair
    assert o["r_claim"] == mle2(Rl, r12).pair


@pytest.fixture(scope="module")
def honest2():
    rng = np.random.default_rng(15)
    A = rng.integers(-400, 400, size=(8, 16))
    B = rng.integers(-400, 400, size=(16, 8))
    chal = inputs.xorshift64_stream(4343, 1024)
    res = orc.prove_layer_fp2(A, B, 7, True, 0, chal)
    res["A"], res["B"] = A, B
    return res, chal


def verify2(res, chal, **over):
    tr = dict(res)
    tabs = {k: np.array(res[k], copy=True) for k in ("A", "B", "Z", "R", "Rm", "Y", "bits")}
    for k, v in over.items():
        if k in tabs:
            tabs[k] = v
        else:
            tr[k] = v
    return orc.verify_layer_fp2(tabs["A"], tabs["B"], tabs["Z"], res["s"], res["relu"], res["mode"], tabs["R"],
                                tabs["Rm"], tabs["Y"], tabs["bits"], tr, chal)[0]


def test_fp2_honest_accepts_and_tampers_reject(honest2):
    res, chal = honest2
    assert verify2(res, chal) == 0
    bump = lambda v, part: ((v[0] + (part == 0)) % P, (v[1] + (part == 1)) % P)
    for key in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim", "range_sum", "bits_claim",
                "r_at", "y_at"):
        for part in (0, 1):
            assert verify2(res, chal, **{key: bump(res[key], part)}) != 0, (key, part)
    for key in ("mm_evals", "rs_evals", "zc_evals"):
        for i in (0, len(res[key]) - 1):
            ev = list(res[key]); ev[i] = bump(ev[i], 1)
            assert verify2(res, chal, **{key: ev}) != 0, key
    # openings: a* -> c a*, b* -> b* / c keeps a* b*; r_at -> -r_at keeps r_at^2
    cst = (2, 3)
    assert verify2(res, chal, a_star=orc.f2mul(res["a_star"], cst),
                   b_star=orc.f2mul(res["b_star"], orc.f2inv(cst))) == 3
    neg = lambda v: ((P - v[0]) % P, (P - v[1]) % P)
    assert verify2(res, chal, r_at=neg(res["r_at"])) == 10
    assert verify2(res, chal, y_at=neg(res["y_at"])) == 10
    Z = res["Z"].copy(); Z[0, 0] += 1
    assert verify2(res, chal, Z=Z) != 0
    b1 = res["bits"].astype(np.int64).copy(); b1[2, 3] ^= 1
    assert verify2(res, chal, bits=b1) != 0


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_fp2_networks_verify(cfg):
    wl = inputs.small(cfg)
    outs = orc.prove_network_fp2(wl)
    chal = orc.fp2_stream(wl)
    cur = 0
    for li, res in enumerate(outs):
        v, cur = orc.verify_layer_fp2(res["A"], wl.layers[li].B, res["Z"], res["s"], res["relu"], res["mode"],
                                      res["R"], res["Rm"], res["Y"], res["bits"], res, chal, cur)
        assert v == 0, (cfg, li)
