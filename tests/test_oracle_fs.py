"""Pins of the oracle's non-interactive protocol (oracle/ra_oracle_fs.c and
the Fiat-Shamir prover / verifier of oracle/ra_oracle_fp2.c), each against
something other than the oracle:
 - SHA-256 against Python's hashlib (FIPS 180-4) at every padding boundary;
 - the Merkle root of the witness tables against its definition written out
   here with hashlib;
 - the transcript's draws against the definition written out here, replayed
   from the proof's own messages in the prover's order;
 - the Fiat-Shamir proof against the interactive prover (already pinned)
   given the challenges the transcript drew;
 - the verifier's accept / reject behaviour.
"""
import hashlib
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2505_17623_amd import inputs

P = (1 << 61) - 1
LABEL = b"range-arithmetic fs v1"


def le(v, n):
    return int(v).to_bytes(n, "little", signed=int(v) < 0)


def f2bytes(pairs):
    return b"".join(int(re).to_bytes(8, "little") + int(im).to_bytes(8, "little") for re, im in pairs)


class Transcript:
    """The draw rule, written from its definition with hashlib."""

    def __init__(self, domain):
        self.S = hashlib.sha256(LABEL + domain).digest()
        self.Q = b""

    def absorb(self, m):
        self.Q += m

    def draw(self):
        self.S = hashlib.sha256(self.S + len(self.Q).to_bytes(4, "little") + self.Q).digest()
        self.Q = b""
        return (int.from_bytes(self.S[:8], "little") % P, int.from_bytes(self.S[8:16], "little") % P)


def root_by_definition(R, Rm, Y, Z, words):
    blobs = [b"".join(le(v, 4) for v in R), b"".join(le(v, 2) for v in Rm), b"".join(le(v, 4) for v in Y),
             b"".join(le(v, 4) for v in Z), b"".join(int(w).to_bytes(8, "little") for w in words)]
    data = b"".join(b + bytes(-len(b) % 1024) for b in blobs)
    dig = [hashlib.sha256(b"\x00" + data[i:i + 1024]).digest() for i in range(0, len(data), 1024)]
    leaves = len(dig)
    while len(dig) > 1:
        dig = [hashlib.sha256(b"\x01" + b"".join(dig[i:i + 4]) + bytes(32 * (4 - len(dig[i:i + 4])))).digest()
               for i in range(0, len(dig), 4)]
    return hashlib.sha256(b"\x02" + leaves.to_bytes(8, "little") + dig[0]).digest()


def test_sha256_matches_hashlib():
    rng = np.random.default_rng(1)
    for n in list(range(0, 130)) + [1025, 4096, 4097]:
        m = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        assert orc.sha256(m) == hashlib.sha256(m).digest(), n


@pytest.mark.parametrize("N", [1, 7, 4096])
def test_witness_root_matches_definition(N):
    rng = np.random.default_rng(N)
    R = rng.integers(-2 ** 31, 2 ** 31, size=N)
    Rm = rng.integers(0, 2 ** 16, size=N)
    Y = rng.integers(0, 2 ** 31, size=N)
    Z = rng.integers(-2 ** 31, 2 ** 31, size=N)
    words = rng.integers(0, 2 ** 63, size=N, dtype=np.uint64)
    assert orc.witness_root(R, Rm, Y, Z, words) == root_by_definition(R, Rm, Y, Z, words)


def test_transcript_draws_match_definition():
    domain = hashlib.sha256(b"pins").digest()
    st, ref = orc.fs_init(domain), Transcript(domain)
    rng = np.random.default_rng(2)
    for step in range(40):
        if step % 3:
            m = rng.integers(0, 256, size=int(rng.integers(0, 200)), dtype=np.uint8).tobytes()
            orc.fs_absorb(st, m)
            ref.absorb(m)
        assert orc.fs_draw(st) == ref.draw()


def small_fs_network(cfg):
    wl = inputs.small(cfg)
    domain = hashlib.sha256(wl.name.encode()).digest()
    pubs = [hashlib.sha256(f"{wl.name}/layer {li}".encode()).digest() for li in range(len(wl.layers))]
    return wl, domain, pubs, orc.prove_network_fs(wl, domain, pubs)


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_draws_follow_the_transcript(cfg):
    """Replay each layer's messages in the prover's order through the
    definition: the challenges must be the ones the prover drew."""
    wl, domain, pubs, res = small_fs_network(cfg)
    T = Transcript(domain)
    for li, r in enumerate(res):
        n, m, k, P = r["n"], r["m"], r["k"], r["P"]
        ln, lm, lk, lP = (n.bit_length() - 1, m.bit_length() - 1, k.bit_length() - 1, P.bit_length() - 1)
        lN = ln + lk
        hdr = b"".join(le(v, 4) for v in (n, m, k, r["s"], r["relu"], r["mode"], r["t"], P))
        root = root_by_definition(r["R"].reshape(-1), r["Rm"].reshape(-1), r["Y"].reshape(-1), r["Z"].reshape(-1),
                                  orc.pack_words(r["bits"]))
        T.absorb(hdr + pubs[li] + root)
        want = [T.draw() for _ in range(ln + lk)]
        for j in range(lm):
            T.absorb(f2bytes(r["mm_evals"][3 * j:3 * j + 3]))
            want.append(T.draw())
        T.absorb(f2bytes([r[x] for x in ("a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim")]))
        want += [T.draw() for _ in range(4 + lP)]
        for j in range(lP + lN):
            T.absorb(f2bytes(r["rs_evals"][4 * j:4 * j + 4]))
            want.append(T.draw())
        T.absorb(f2bytes([r["bits_claim"]]))
        if r["relu"]:
            for j in range(lN):
                T.absorb(f2bytes(r["zc_evals"][4 * j:4 * j + 4]))
                want.append(T.draw())
            T.absorb(f2bytes([r["r_at"], r["y_at"]]))
        assert r["drawn"] == want, f"layer {li}"


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_fs_proof_is_the_interactive_proof_at_its_challenges(cfg):
    """Given the challenges the transcript drew (as the F_p stream in pairs),
    the interactive prover produces the same transcript and tables."""
    wl, domain, pubs, res = small_fs_network(cfg)
    for li, r in enumerate(res):
        stream = np.array([c for pair in r["drawn"] for c in pair], dtype=np.uint64)
        o = orc.prove_layer_fp2(r["A"], wl.layers[li].B, r["s"], r["relu"], r["mode"], stream, 0)
        for key in ("t", "P", "mm_evals", "rs_evals", "zc_evals") + orc.F2_SCALARS:
            assert o[key] == r[key], (li, key)
        for key in ("C", "R", "Rm", "Y", "Z", "bits"):
            assert np.array_equal(o[key], r[key]), (li, key)
        assert o["cursor"] == len(stream)


def verify_all(wl, domain, pubs, res, layers=None):
    st = orc.fs_init(domain)
    for li, r in enumerate(res):
        L = layers[li] if layers else r
        v = orc.verify_layer_fs(L["A"], wl.layers[li].B, L["Z"], r["s"], r["relu"], r["mode"], L["R"], L["Rm"],
                                L["Y"], L["bits"].astype(np.int64), L["tr"] if layers else r, st, pubs[li])
        if v:
            return v, li
    return 0, 0


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_fs_verifier_accepts(cfg):
    wl, domain, pubs, res = small_fs_network(cfg)
    assert verify_all(wl, domain, pubs, res) == (0, 0)


def test_fs_verifier_rejects():
    wl, domain, pubs, res = small_fs_network(2)
    assert verify_all(wl, domain, pubs, res) == (0, 0)

    def with_layer(li, tr=None, **tables):
        layers = []
        for i, r in enumerate(res):
            L = dict(A=r["A"], Z=r["Z"], R=r["R"], Rm=r["Rm"], Y=r["Y"], bits=r["bits"], tr=r)
            if i == li:
                L.update(tables)
                if tr is not None:
                    L["tr"] = tr
            layers.append(L)
        return layers

    # another domain or another public digest: other challenges, the proof fails
    assert verify_all(wl, hashlib.sha256(b"other").digest(), pubs, res)[0] != 0
    assert verify_all(wl, domain, [pubs[0], bytes(32), pubs[2]], res)[0] != 0
    # a changed round word (any instance), final value or claim
    r1 = res[1]
    for key, idx in (("mm_evals", 0), ("rs_evals", 5), ("zc_evals", 2), ("a_star", None), ("bits_claim", None)):
        if idx is None:
            re, im = r1[key]
            tr = dict(r1, **{key: (re, (im + 1) % P)})
        else:
            ev = list(r1[key])
            re, im = ev[idx]
            ev[idx] = ((re + 1) % P, im)
            tr = dict(r1, **{key: ev})
        v, li = verify_all(wl, domain, pubs, res, with_layer(1, tr=tr))
        assert v != 0 and li == 1, key
    # a witness entry changed after the proof: its root, hence every
    # challenge, differs
    R = r1["R"].copy()
    R.flat[3] += 1
    v, li = verify_all(wl, domain, pubs, res, with_layer(1, R=R))
    assert v != 0 and li == 1
    bits = r1["bits"].copy()
    bits[0, 0] ^= 1
    v, li = verify_all(wl, domain, pubs, res, with_layer(1, bits=bits))
    assert v != 0 and li == 1
