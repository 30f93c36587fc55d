"""Pins of the oracle's gather link (oracle/ra_oracle.c, orc_link_prove /
orc_link_verify): the reduction of the next layer's claim A~(z), for an input
A that gathers the previous output Z (im2col, flattening), to claims on
Z~ and W~_z at a fresh point.  Each pin checks against something other than
the oracle: the multilinear extension of the gathered matrix itself (Eq. (1),
by brute force), brute-force hypercube sums of the round polynomials
(Sec. II-D), the identity gather (a closed form), and the verifier's accept /
reject behaviour with tampers that keep the earlier checks true."""
import numpy as np
import pytest

import brute
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

P = (1 << 61) - 1


def tiny_case(rng, nz=16, na=32, pad=0.25):
    Z = rng.integers(-500, 500, size=nz)
    src = rng.integers(0, nz, size=na)           # repeated sources, as im2col has
    src[rng.random(na) < pad] = -1               # zero padding
    return Z, src


def gathered(Z, src):
    return [int(Z[s]) if s >= 0 else 0 for s in src]


def test_link_claim_and_rounds_brute_force():
    rng = np.random.default_rng(21)
    Z, src = tiny_case(rng)
    vz, va = 4, 5
    chal = inputs.xorshift64_stream(77, 64)
    z = [int(x) for x in inputs.xorshift64_stream(78, va)]
    res = orc.prove_link(Z, src, z, chal, 0)
    A = gathered(Z, src)
    assert res["claim"] == brute.mle(A, z)                         # A~(z), Eq. (1) on the gathered matrix
    ys = [int(x) for x in chal[:vz]]

    def W_at(pt):  # W~_z(pt) = sum_a eq(z, a) eq(pt, src[a])
        return sum(brute.eq_point(z, brute.bits_msb(a, va)) * brute.eq_point(pt, brute.bits_msb(int(s), vz))
                   for a, s in enumerate(src) if s >= 0) % P

    def f(pt):
        return brute.mle([int(x) for x in Z], pt) * W_at(pt) % P

    g = brute.round_polys(vz, 2, f, ys)
    assert [x for r in g for x in r] == res["evals"]
    assert res["z_at"] == brute.mle([int(x) for x in Z], ys)
    assert res["w_at"] == W_at(ys)
    assert res["cursor"] == vz


def test_identity_gather_is_the_mle_of_z():
    """src = identity: A = Z, so the claim is Z~(z) and W_z = eq(z, .)."""
    rng = np.random.default_rng(22)
    Z = rng.integers(-10 ** 6, 10 ** 6, size=64)
    z = [int(x) for x in inputs.xorshift64_stream(5, 6)]
    chal = inputs.xorshift64_stream(6, 6)
    res = orc.prove_link(Z, np.arange(64), z, chal, 0)
    assert res["claim"] == brute.mle([int(x) for x in Z], z)
    ys = [int(x) for x in chal]
    assert res["w_at"] == brute.eq_point(z, ys)                    # eq(z, y*), a closed form


def test_link_of_a_small_cnn_matches_the_gathered_input():
    """Every link of the small CNN: the claim equals A~(z) of the layer input
    the workload builds (im2col / flatten of the previous output)."""
    wl = inputs.small(4)
    res = orc.prove_network(wl, links=True)
    cursor_seen = 0
    for li in range(1, len(wl.layers)):
        r = res[li]
        assert "link" in r
        A = wl.layer_input(li, res[li - 1]["Z"])
        assert np.array_equal(A, r["A"])
        want = orc.mle_int(A.reshape(-1), r["link_point"])
        assert r["link"]["claim"] == want == r["a_star"]
        v, _ = orc.verify_link(res[li - 1]["Z"], wl.link_map(li), r["link_point"], r["a_star"], r["link"],
                               wl.challenges, r["link"]["cursor"] - (len(r["link"]["evals"]) // 3))
        assert v == 0
        cursor_seen = r["cursor"]
    assert cursor_seen == res[-1]["cursor"]


@pytest.fixture(scope="module")
def honest_link():
    rng = np.random.default_rng(23)
    Z, src = tiny_case(rng, nz=64, na=128)
    z = [int(x) for x in inputs.xorshift64_stream(9, 7)]
    chal = inputs.xorshift64_stream(10, 32)
    res = orc.prove_link(Z, src, z, chal, 0)
    return Z, src, z, chal, res


def test_link_verifier_accepts(honest_link):
    Z, src, z, chal, res = honest_link
    assert orc.verify_link(Z, src, z, res["claim"], res, chal, 0) == (0, 6)


def test_link_verifier_rejects(honest_link):
    Z, src, z, chal, res = honest_link
    a = res["claim"]

    def v(link=res, Zv=Z, srcv=src, a_star=a):
        return orc.verify_link(Zv, srcv, z, a_star, link, chal, 0)[0]

    for i in range(len(res["evals"])):                              # every round word
        ev = list(res["evals"])
        ev[i] = (ev[i] + 1) % P
        assert v(dict(res, evals=ev)) == 15
    assert v(a_star=(a + 1) % P) == 15                              # a claim other than the layer's a*
    assert v(dict(res, z_at=(res["z_at"] + 1) % P)) == 15
    # the final product kept: z_at scaled by 2, w_at by 1/2 -> only the Z opening fails
    half = (P + 1) // 2
    assert v(dict(res, z_at=2 * res["z_at"] % P, w_at=res["w_at"] * half % P)) == 15
    Z2 = np.array(Z)
    Z2[3] += 1                                                       # a different previous output
    assert v(Zv=Z2) == 15
    # a different public gather map: the chain and the Z opening hold, only W~ fails
    src2 = np.array(src)
    j = int(np.flatnonzero(src2 >= 0)[0])
    src2[j] = (src2[j] + 1) % len(Z)
    assert v(srcv=src2) == 15
