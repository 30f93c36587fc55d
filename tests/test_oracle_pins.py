"""Pins of the CPU oracle against what the paper and plain mathematics fix.

Each test ties one oracle function to something other than the oracle: Python
big-integer arithmetic, the brute-force formulas of tests/brute.py (Eq. (1),
direct hypercube sums), the worked example of Sec. III-A-1, Theorem A.1 by
enumeration, closed forms (Eq. (4), recomposition sums), and the soundness
statements of Sec. IV (tampered transcripts and tables are rejected).
"""
import json
import os
import random

import numpy as np
import pytest

import brute
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

P = orc.P61
GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _built():
    orc.build(force=False)


def rnd_field(rng, n):
    return [rng.randrange(P) for _ in range(n)]


# --- field --------------------------------------------------------------
def test_field_ops_match_python_integers():
    rng = random.Random(1)
    edges = [0, 1, 2, P - 1, P - 2, (1 << 60), (1 << 32) - 1, 1 << 32]
    vals = edges + rnd_field(rng, 200)
    for a in vals:
        for b in vals[:20] + rnd_field(rng, 5):
            assert orc.fmul(a, b) == a * b % P
            assert orc.fadd(a, b) == (a + b) % P
            assert orc.fsub(a, b) == (a - b) % P
    for z in [0, 1, -1, -(1 << 40), (1 << 62), -(1 << 62), (1 << 63) - 1, -(1 << 63)]:
        assert orc.fint(z) == z % P


# --- multilinear extensions ----------------------------------------------
def test_chi_vector_matches_eq1_product():
    rng = random.Random(2)
    for v in range(0, 8):
        z = rnd_field(rng, v)
        vec = orc.chi_vector(z)
        for y in range(1 << v):
            want = brute.eq_point(z, brute.bits_msb(y, v))
            assert int(vec[y]) == want
            assert orc.chi_at(z, y) == want


def test_mle_matches_eq1_and_interpolates_hypercube():
    rng = random.Random(3)
    for v in range(0, 7):
        tab = [rng.randrange(-2 ** 40, 2 ** 40) for _ in range(1 << v)]
        z = rnd_field(rng, v)
        assert orc.mle_int(tab, z) == brute.mle(tab, z)
        ft = [t % P for t in tab]
        assert orc.mle_field(ft, z) == brute.mle(tab, z)
        for y in range(1 << v):                       # agrees with e on {0,1}^v
            assert orc.mle_int(tab, brute.bits_msb(y, v)) == tab[y] % P


def test_mle_is_multilinear():
    # linear in each variable: e~(.., 2, ..) = 2 e~(.., 1, ..) - e~(.., 0, ..)
    rng = random.Random(4)
    v = 5
    tab = [rng.randrange(-1000, 1000) for _ in range(1 << v)]
    z = rnd_field(rng, v)
    for i in range(v):
        pts = [list(z) for _ in range(3)]
        for X in range(3):
            pts[X][i] = X
        e = [orc.mle_int(tab, p) for p in pts]
        assert e[2] == (2 * e[1] - e[0]) % P


def test_worked_index_example():
    g = json.load(open(os.path.join(GOLD, "worked_example_index.json")))
    rng = np.random.default_rng(5)
    A = rng.integers(0, 50, size=(g["rows"], g["cols"]))
    A[g["row"], g["col"]] = g["value"]
    point = g["row_bits"] + g["col_bits"]
    assert orc.mle_int(A, point) == g["value"]
    # an LSB-first or column-major reading would pick a different entry
    assert A[0, 1] != g["value"] and A[2, 0] != g["value"]


# --- rounding, t, ReLU -----------------------------------------------------
def small_layer(rng, n, m, k, lo, hi, s, relu, mode=0):
    A = rng.integers(lo, hi, size=(n, m))
    B = rng.integers(lo, hi, size=(m, k))
    chal = inputs.xorshift64_stream(12345 + n + m + k + s, 512)
    return A, B, orc.prove_layer(A, B, s, relu, mode, chal), chal


def test_rounding_operator_and_remainder_interval():
    rng = np.random.default_rng(6)
    for s in (1, 3, 8, 12):
        A, B, res, _ = small_layer(rng, 8, 8, 8, -300, 300, s, True)
        C = A.astype(object) @ B.astype(object)
        assert np.array_equal(res["C"], C.astype(np.int64))
        for c, r, rm in zip(C.reshape(-1), res["R"].reshape(-1), res["Rm"].reshape(-1)):
            assert r == brute.rounding(int(c), s)
            e = int(rm) - (1 << (s - 1))
            assert -(1 << (s - 1)) <= e < (1 << (s - 1))          # Sec. III-A-2 interval
            assert int(c) == (1 << s) * int(r) + e                   # C = 2^s C' + E
            assert abs(2 * int(c) - (int(r) << (s + 1))) <= (1 << s)  # nearest: |c/2^s - r| <= 1/2


def test_rounding_exhaustive_small_range():
    # every integer in [-2^12, 2^12] through a 1x1x1 layer with B = 1
    for s in (1, 2, 5, 8):
        xs = np.arange(-(1 << 12), (1 << 12) + 1)
        for x in xs[:: 97]:
            res = orc.prove_layer(np.array([[x]]), np.array([[1]]), s, False, 0,
                                  inputs.xorshift64_stream(7, 64))
            assert int(res["R"][0, 0]) == brute.rounding(int(x), s)
            q, r = divmod(int(x), 1 << s)                             # floor mode
            res2 = orc.prove_layer(np.array([[x]]), np.array([[1]]), s, False, 1,
                                   inputs.xorshift64_stream(7, 64))
            assert int(res2["R"][0, 0]) == q and int(res2["Rm"][0, 0]) == r


def test_t_is_least_and_relu_output():
    rng = np.random.default_rng(8)
    A, B, res, _ = small_layer(rng, 8, 16, 8, -500, 500, 6, True)
    R = res["R"].astype(np.int64)
    t = res["t"]
    assert np.all((R >= -(1 << (t + 1))) & (R < (1 << (t + 1))))
    if t > 0:
        assert not np.all((R >= -(1 << t)) & (R < (1 << t)))
    assert np.array_equal(res["Y"], np.abs(R))
    assert np.array_equal(res["Z"], np.maximum(R, 0))
    assert np.array_equal(2 * res["Z"], R + np.abs(R))                # ReLU = (x + |x|)/2
    Q = 6 + (t + 2) * 2
    assert res["P"] == inputs.next_pow2(Q) and orc.plane_count(6, t, True) == Q


def test_bit_table_recomposes_values():
    rng = np.random.default_rng(9)
    A, B, res, _ = small_layer(rng, 4, 8, 8, -200, 200, 5, True)
    t, bits = res["t"], res["bits"].astype(np.int64)
    s = 5
    w = lambda lo, cnt: sum(bits[lo + b] << b for b in range(cnt))
    assert np.array_equal(w(0, s), res["Rm"].reshape(-1))
    assert np.array_equal(w(s, t + 2), res["R"].reshape(-1) + (1 << (t + 1)))
    assert np.array_equal(w(s + t + 2, t + 2), res["Y"].reshape(-1))
    assert not bits[s + 2 * t + 4:].any()


def test_theorem_a1_enumeration():
    g = json.load(open(os.path.join(GOLD, "theorem_a1_small.json")))
    s, t = g["s"], g["t"]

    def unique(p):
        # for every field element a, at most one (a', e) with a = e + 2^s a'
        # (mod p), -2^(t+1) <= a' < 2^(t+1), -2^(s-1) <= e < 2^(s-1)
        seen = {}
        for ap in range(-(1 << (t + 1)), 1 << (t + 1)):
            for e in range(-(1 << (s - 1)), 1 << (s - 1)):
                a = (e + (1 << s) * ap) % p
                if a in seen:
                    return False
                seen[a] = (ap, e)
        return True

    primes = [q for q in range(3, 64) if all(q % d for d in range(2, q))]
    for q in primes:
        if q.bit_length() >= s + t + 3:
            assert unique(q), q
    assert all(q in primes and unique(q) for q in g["unique_for_primes"])
    assert not all(unique(q) for q in primes if q.bit_length() == s + t + 2)


def test_field_guard_s_t():
    chal = inputs.xorshift64_stream(99, 512)
    # s = 30: R = 2^28 needs t = 28 (s + t + 3 = 61, allowed); R = 2^29 needs t = 29 (62, refused)
    ok = orc.prove_layer(np.array([[1 << 29]]), np.array([[1 << 29]]), 30, False, 0, chal)
    assert ok["t"] == 28
    with pytest.raises(orc.OracleError) as e:
        orc.prove_layer(np.array([[1 << 30]]), np.array([[1 << 29]]), 30, False, 0, chal)
    assert e.value.code == -3
    with pytest.raises(orc.OracleError) as e:             # explicit t too small
        orc.prove_layer(np.array([[1 << 20]]), np.array([[1]]), 4, False, 0, chal, t_in=10)
    assert e.value.code == -4


# --- the sum-checks against brute force ------------------------------------
def challenge_layout(res, chal, cursor=0):
    n, m, k, P_ = res["n"], res["m"], res["k"], res["P"]
    ln, lm, lk, lP = (x.bit_length() - 1 for x in (n, m, k, P_))
    lN = ln + lk
    c = [int(x) for x in chal[cursor:]]
    d = {}
    d["r1"], c = c[:ln], c[ln:]
    d["r2"], c = c[:lk], c[lk:]
    d["rho"], c = c[:lm], c[lm:]
    d["lam"], c = c[:3], c[3:]
    d["mu"], c = c[0], c[1:]
    d["tau_p"], c = c[:lP], c[lP:]
    d["sigma"], c = c[:lP + lN], c[lP + lN:]
    d["rho2"] = c[:lN] if res["relu"] else []
    return d, ln, lm, lk, lP, lN


def test_matmul_sumcheck_brute_force_and_eq4():
    rng = np.random.default_rng(10)
    A, B, res, chal = small_layer(rng, 4, 8, 4, -50, 50, 3, False)
    d, ln, lm, lk, lP, lN = challenge_layout(res, chal)
    Af = [int(x) for x in A.reshape(-1)]
    Bf = [int(x) for x in B.reshape(-1)]
    # Eq. (4): c0 = C~(r1, r2) for the exact integer product
    C = (A.astype(object) @ B.astype(object)).reshape(-1)
    assert res["c0"] == brute.mle(list(C), d["r1"] + d["r2"])

    def gamma(pt):
        return brute.mle(Af, d["r1"] + pt) * brute.mle(Bf, pt + d["r2"]) % P

    g = brute.round_polys(lm, 2, gamma, d["rho"])
    assert [x for r in g for x in r] == res["mm_evals"]
    assert res["a_star"] == brute.mle(Af, d["r1"] + d["rho"])
    assert res["b_star"] == brute.mle(Bf, d["rho"] + d["r2"])
    # rounding link: C = 2^s R + Rm - 2^(s-1) in the field at (r1, r2)
    s = 3
    assert res["c0"] == ((1 << s) * res["r_claim"] + res["rm_claim"] - (1 << (s - 1))) % P


def plane_weights(res, lam, s, t, relu):
    W = [0] * res["P"]
    q = 0
    for b in range(s):
        W[q] = lam[0] * (1 << b) % P; q += 1
    for b in range(t + 2):
        W[q] = lam[1] * (1 << b) % P; q += 1
    if relu:
        for b in range(t + 2):
            W[q] = lam[2] * (1 << b) % P; q += 1
    return W


@pytest.mark.parametrize("relu", [False, True])
def test_range_and_relu_sumchecks_brute_force(relu):
    rng = np.random.default_rng(11 + relu)
    s = 1
    A = rng.integers(-1, 2, size=(2, 4))
    B = rng.integers(-1, 2, size=(4, 2))
    chal = inputs.xorshift64_stream(777 + relu, 256)
    res = orc.prove_layer(A, B, s, relu, 0, chal)
    d, ln, lm, lk, lP, lN = challenge_layout(res, chal)
    t = res["t"]
    N = 4
    bits = [int(b) for b in res["bits"].reshape(-1)]
    W = plane_weights(res, d["lam"], s, t, relu)
    r12 = d["r1"] + d["r2"]
    tau = d["tau_p"] + r12
    mu = d["mu"]
    v = lP + lN
    assert v <= 8

    def f_range(pt):
        b = brute.mle(bits, pt)
        eqt = brute.eq_point(tau, pt)
        wx = brute.mle(W, pt[:lP]) * brute.eq_point(r12, pt[lP:]) % P
        return (eqt * b % P * (b - 1) + mu * wx % P * b) % P

    g = brute.round_polys(v, 3, f_range, d["sigma"])
    assert [x for r in g for x in r] == res["rs_evals"]
    assert res["bits_claim"] == brute.mle(bits, d["sigma"])
    # claimed sum: the hypercube sum equals mu (l1 Rm~ + l2 (R~ + 2^(t+1)) + l3 Y~)
    total = sum(f_range(brute.bits_msb(y, v)) for y in range(1 << v)) % P
    lam = d["lam"]
    H = lam[0] * brute.mle(list(res["Rm"].reshape(-1)), r12) + \
        lam[1] * (brute.mle(list(res["R"].reshape(-1)), r12) + (1 << (t + 1)))
    if relu:
        H += lam[2] * brute.mle(list(res["Y"].reshape(-1)), r12)
    assert total == mu * H % P == res["range_sum"]
    assert (g[0][0] + g[0][1]) % P == total
    if relu:
        Rl = [int(x) for x in res["R"].reshape(-1)]
        Yl = [int(x) for x in res["Y"].reshape(-1)]

        def f_relu(pt):
            r, y = brute.mle(Rl, pt), brute.mle(Yl, pt)
            return brute.eq_point(r12, pt) * (r * r - y * y) % P

        gz = brute.round_polys(lN, 3, f_relu, d["rho2"])
        assert [x for r in gz for x in r] == res["zc_evals"]
        assert res["r_at"] == brute.mle(Rl, d["rho2"]) and res["y_at"] == brute.mle(Yl, d["rho2"])
    else:
        assert res["zc_evals"] == []


def test_interp_is_lagrange():
    rng = random.Random(13)
    for deg in (1, 2, 3):
        coef = rnd_field(rng, deg + 1)
        poly = lambda x: sum(c * pow(x, i, P) for i, c in enumerate(coef)) % P
        ev = [poly(i) for i in range(deg + 1)]
        x = rng.randrange(P)
        assert orc.interp(ev, x) == poly(x) == brute.lagrange_eval(ev, x)


# --- completeness and soundness (Sec. II-F, Sec. IV) -----------------------
def verify(res, chal, cursor=0, **over):
    tr = dict(res)
    tabs = {k: np.array(res[k], copy=True) for k in ("A", "B", "Z", "R", "Rm", "Y", "bits")}
    for k, v in over.items():
        if k in tabs:
            tabs[k] = v
        else:
            tr[k] = v
    return orc.verify_layer(tabs["A"], tabs["B"], tabs["Z"], res["s"], res["relu"], res["mode"],
                            tabs["R"], tabs["Rm"], tabs["Y"], tabs["bits"], tr, chal, cursor)[0]


@pytest.fixture(scope="module")
def honest():
    rng = np.random.default_rng(14)
    A = rng.integers(-400, 400, size=(8, 16))
    B = rng.integers(-400, 400, size=(16, 8))
    chal = inputs.xorshift64_stream(4242, 512)
    res = orc.prove_layer(A, B, 7, True, 0, chal)
    res["A"], res["B"] = A, B
    return res, chal


def test_honest_transcripts_accept(honest):
    res, chal = honest
    assert verify(res, chal) == 0
    for mode in (0, 1):
        for relu in (False, True):
            rng = np.random.default_rng(20 + mode * 2 + relu)
            A = rng.integers(-900, 900, size=(4, 8))
            B = rng.integers(-900, 900, size=(8, 16))
            chal2 = inputs.xorshift64_stream(31 + mode, 512)
            r = orc.prove_layer(A, B, 9, relu, mode, chal2)
            r["A"], r["B"] = A, B
            assert verify(r, chal2) == 0


def test_network_chain_accepts():
    wl = inputs.small(2)
    outs = orc.prove_network(wl)
    cur = 0
    for li, res in enumerate(outs):
        res["B"] = wl.layers[li].B
        v, cur = orc.verify_layer(res["A"], res["B"], res["Z"], res["s"], res["relu"], res["mode"],
                                  res["R"], res["Rm"], res["Y"], res["bits"], res, wl.challenges, cur)
        assert v == 0
        if li + 1 < len(outs):
            assert np.array_equal(outs[li + 1]["A"], res["Z"])


def test_tampered_output_rejected(honest):
    res, chal = honest
    Z = res["Z"].copy(); Z[1, 2] += 1
    assert verify(res, chal, Z=Z) != 0


def test_tampered_rounding_rejected(honest):
    res, chal = honest
    s = res["s"]
    # R off by one with Z kept consistent: the rounding link fails
    R = res["R"].copy(); R[0, 0] += 1
    Y = np.abs(R); Z = np.maximum(R, 0)
    assert verify(res, chal, R=R, Y=Y, Z=Z) != 0
    # remainder out of range with the linear relation C = 2^s R + E kept
    R2 = res["R"].copy(); Rm2 = res["Rm"].copy()
    R2[2, 3] -= 1; Rm2[2, 3] += 1 << s
    assert verify(res, chal, R=R2, Rm=Rm2, Y=np.abs(R2), Z=np.maximum(R2, 0)) != 0


def test_tampered_relu_sign_rejected(honest):
    res, chal = honest
    R = res["R"]
    neg = np.argwhere(R < 0)[0]
    Y = res["Y"].copy(); Y[tuple(neg)] = R[tuple(neg)]           # "|x|" = x for a negative x
    Z = (R + Y) // 2
    assert verify(res, chal, Y=Y, Z=Z) != 0


def test_tampered_bits_rejected(honest):
    res, chal = honest
    bits = res["bits"].astype(np.int64)
    b1 = bits.copy(); b1[3, 5] ^= 1
    assert verify(res, chal, bits=b1) != 0
    # non-boolean digit that still recomposes: Rm bit0 := bit0 + 2, bit1 := bit1 - 1
    x = int(np.argwhere(bits[1] == 1)[0][0])
    b2 = bits.copy(); b2[1, x] -= 1; b2[0, x] += 2
    assert verify(res, chal, bits=b2) != 0


def test_tampered_transcript_words_rejected(honest):
    res, chal = honest
    for key in ("mm_evals", "rs_evals", "zc_evals"):
        for i in (0, len(res[key]) // 2, len(res[key]) - 1):
            ev = list(res[key]); ev[i] = (ev[i] + 1) % P
            assert verify(res, chal, **{key: ev}) != 0, (key, i)
    for key in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
                "bits_claim", "r_at", "y_at"):
        assert verify(res, chal, **{key: (res[key] + 1) % P}) != 0, key
    assert verify(res, chal, t=res["t"] + 1) != 0
    assert verify(res, chal, c0=res["c0"] + P) != 0                  # non-canonical word


def test_openings_rejected_when_earlier_identities_hold(honest):
    """Tampers that keep every identity before an opening true, so only the
    opening of the final claims against the tables can reject them (Sec. IV:
    the final sum-check claims are bound to the committed, here opened,
    tables).  a* -> 2 a*, b* -> b* / 2 keeps a* b*, so the matrix chain and
    its final identity hold and check 3 must fail; r_at -> -r_at (or y_at ->
    -y_at) keeps r_at^2 - y_at^2, so the ReLU chain holds and check 10 must
    fail."""
    res, chal = honest
    inv2 = pow(2, P - 2, P)
    assert verify(res, chal, a_star=2 * res["a_star"] % P, b_star=res["b_star"] * inv2 % P) == 3
    assert verify(res, chal, r_at=(P - res["r_at"]) % P) == 10
    assert verify(res, chal, y_at=(P - res["y_at"]) % P) == 10
    # a public input entry changed: only the opening of a* sees it
    A = np.array(res["A"], copy=True); A[1, 3] += 1
    assert verify(res, chal, A=A) == 3
    B = np.array(res["B"], copy=True); B[2, 0] -= 1
    assert verify(res, chal, B=B) == 3


def test_challenge_stream_is_xorshift64():
    """The seeded challenge stream is Marsaglia's xor64 generator (shifts 13,
    7, 17) reduced mod p: its raw outputs from the example state of that
    paper, reduced, are the first challenges (tests/golden/xorshift64_marsaglia.json)."""
    g = json.load(open(os.path.join(GOLD, "xorshift64_marsaglia.json")))
    got = inputs.xorshift64_stream(g["seed"], len(g["outputs"]))
    assert [int(x) for x in got] == [o % P for o in g["outputs"]]
    assert all(int(x) < P for x in inputs.xorshift64_stream(12345, 2000))
