"""The GPU's non-interactive proofs (ra_prove_layer_fs: Fiat-Shamir over
F_{p^2}, the transcript hashed on the device) against the oracle, through the
C ABI: every transcript word, every witness table and the witness tables'
Merkle root bit-identical, on the small workloads, edge shapes and the full
workloads (tests/golden/full_fs_cfg<N>.json, written by make_golden.py --fs,
which calls only the oracle); both verifiers on the GPU's proofs."""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2505_17623_amd import inputs

pytestmark = pytest.mark.gpu
P61 = (1 << 61) - 1
GOLD = os.path.join(os.path.dirname(__file__), "golden")
KEYS = ["t", "P", "c0", "mm_evals", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
        "range_sum", "rs_evals", "bits_claim", "zc_evals", "r_at", "y_at"]


@pytest.fixture(scope="module")
def ra():
    from paper_2505_17623_amd import ra as ra_mod
    ra_mod.lib()
    assert torch.cuda.is_available()
    return ra_mod


def as_pairs(v):
    if isinstance(v, (list, tuple)) and v and isinstance(v[0], (list, tuple)):
        return [(int(a), int(b)) for a, b in v]
    if isinstance(v, (list, tuple)) and len(v) == 2:
        return [(int(v[0]), int(v[1]))]
    if isinstance(v, (list, tuple)):
        return []
    return [int(v)]


def diff(tr, want):
    return [k for k in KEYS if as_pairs(tr[k]) != as_pairs(want[k])]


def compare(ra, g, o, label):
    bad = diff(g["transcript"], o)
    assert not bad, f"{label}: transcript words differ in {bad}"
    assert np.array_equal(g["C"].cpu().numpy(), o["C"]), label
    for key in ("R", "Y", "Z"):
        assert np.array_equal(g[key].cpu().numpy().astype(np.int64), o[key]), (label, key)
    assert np.array_equal(g["Rm"].cpu().numpy().view(np.uint16).astype(np.int64), o["Rm"]), label
    assert np.array_equal(ra.unpack_bits(g["bits"].cpu().numpy(), g["transcript"]["P"]), o["bits"]), label
    root = orc.witness_root(o["R"], o["Rm"], o["Y"], o["Z"], orc.pack_words(o["bits"]))
    assert g["root"] == root, label


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_fs_network_matches_oracle(ra, cfg):
    wl = inputs.small(cfg)
    domain, pubs = wl.fs_inputs()
    want = orc.prove_network_fs(wl, domain, pubs)
    got = ra.prove_network_fp2(ra.Context(fs_domain=domain), wl, pubs=pubs)
    for li, (g, o) in enumerate(zip(got, want)):
        compare(ra, g, o, f"cfg{cfg} L{li}")


# (n, m, k, s, relu, mode): degenerate instances (no matrix rounds, N = 1,
# N = 2), no ReLU, several blocks per round
SHAPES = [(1, 1, 1, 3, True, 0), (1, 1, 2, 3, True, 1), (2, 1, 4, 2, True, 1), (1, 8, 1, 4, False, 0),
          (4, 2, 1, 5, True, 0), (128, 64, 128, 11, True, 0), (256, 8, 512, 12, True, 1), (32, 32, 64, 6, False, 1)]


@pytest.mark.parametrize("n,m,k,s,relu,mode", SHAPES)
def test_fs_layer_shapes(ra, n, m, k, s, relu, mode):
    rng = np.random.default_rng(n * 131 + m * 7 + k)
    A = rng.integers(-3000, 3000, size=(n, m)).astype(np.int16)
    B = rng.integers(-3000, 3000, size=(m, k)).astype(np.int16)
    domain = hashlib.sha256(f"shape {n} {m} {k}".encode()).digest()
    pub = hashlib.sha256(b"pub").digest()
    o = orc.prove_layer_fs(A, B, s, relu, mode, orc.fs_init(domain), pub)
    g = ra.prove_layer_fp2(ra.Context(fs_domain=domain), torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(),
                           s, relu, mode, pub=pub)
    compare(ra, g, o, f"{n}x{m}x{k}")


def test_fs_given_t_and_int32(ra):
    rng = np.random.default_rng(3)
    A = rng.integers(-(2 ** 16), 2 ** 16, size=(32, 64)).astype(np.int32)
    B = rng.integers(-(2 ** 10), 2 ** 10, size=(64, 16)).astype(np.int16)
    domain, pub = hashlib.sha256(b"t").digest(), bytes(32)
    o = orc.prove_layer_fs(A, B, 12, True, 0, orc.fs_init(domain), pub)
    o2 = orc.prove_layer_fs(A, B, 12, True, 0, orc.fs_init(domain), pub, t_in=o["t"] + 2)
    for want, t in ((o, -1), (o2, o["t"] + 2)):
        g = ra.prove_layer_fp2(ra.Context(fs_domain=domain), torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(),
                               12, True, 0, t, pub=pub)
        compare(ra, g, want, f"t={t}")


def test_fs_refusals(ra):
    A = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    B = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    with pytest.raises(ra.RAError) as e:                      # a context without a transcript
        ra.prove_layer_fp2(ra.Context(seed=5), A, B, 4, True, 0, pub=bytes(32))
    assert e.value.code == -7
    with pytest.raises(ra.RAError) as e:                      # the stream calls on a transcript context
        ra.prove_layer_fp2(ra.Context(fs_domain=bytes(32)), A, B, 4, True, 0)
    assert e.value.code == -5
    with pytest.raises(ra.RAError) as e:                      # a given t that R does not fit
        ra.prove_layer_fp2(ra.Context(fs_domain=bytes(32)), A, B, 4, True, 0, t=3, pub=bytes(32))
    assert e.value.code == -4


def abi_layers(ra, wl, got):
    return [dict(A=g["A"].cpu().numpy(), B=wl.layers[li].B, Z=g["Z"].cpu().numpy(), R=g["R"].cpu().numpy(),
                 Rm=g["Rm"].cpu().numpy(), Y=g["Y"].cpu().numpy(), bits=g["bits"].cpu().numpy(),
                 transcript=g["transcript"], chained=li > 0 and wl.links[li] is None) for li, g in enumerate(got)]


@pytest.mark.parametrize("cfg", [2, 4, 5])
def test_fs_proofs_verify(ra, cfg):
    """The GPU's non-interactive proofs pass the library's and the oracle's
    verifiers; a changed round word or witness entry is rejected."""
    wl = inputs.small(cfg)
    domain, pubs = wl.fs_inputs()
    got = ra.prove_network_fp2(ra.Context(fs_domain=domain), wl, pubs=pubs)
    layers = abi_layers(ra, wl, got)
    assert ra.ra_verify_fs(domain, pubs, layers) == (0, 0)
    st = orc.fs_init(domain)
    for li, L in enumerate(layers):
        tr = L["transcript"]
        planes = ra.unpack_bits(L["bits"], tr["P"]).astype(np.int64)
        assert orc.verify_layer_fs(L["A"], L["B"], L["Z"], tr["s"], tr["relu"], tr["mode"], L["R"],
                                   L["Rm"].view(np.uint16), L["Y"], planes, tr, st, pubs[li]) == 0
    last = len(layers) - 1
    tr = layers[last]["transcript"]
    ev = list(tr["rs_evals"])
    ev[0] = ((ev[0][0] + 1) % P61, ev[0][1])
    changed = [dict(L) for L in layers]
    changed[last] = dict(changed[last], transcript=dict(tr, rs_evals=ev))
    v, li = ra.ra_verify_fs(domain, pubs, changed)
    assert v != 0 and li == last
    R = layers[0]["R"].copy()
    R.flat[1] += 1
    changed = [dict(L) for L in layers]
    changed[0] = dict(changed[0], R=R)
    v, li = ra.ra_verify_fs(domain, pubs, changed)
    assert v != 0 and li == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_fs_full_workload_matches_oracle(ra, cfg):
    gold = json.load(open(os.path.join(GOLD, f"full_fs_cfg{cfg}.json")))
    gold_fp = json.load(open(os.path.join(GOLD, f"full_cfg{cfg}.json")))
    wl = inputs.workload(cfg, "full")
    domain, pubs = wl.fs_inputs()
    got = ra.prove_network_fp2(ra.Context(fs_domain=domain), wl, ts=[o["transcript"]["t"] for o in gold["layers"]],
                               bufs=[], pubs=pubs)
    for li, (g, o, ofp) in enumerate(zip(got, gold["layers"], gold_fp["layers"])):
        bad = diff(g["transcript"], o["transcript"])
        assert not bad, f"config {cfg} layer {li}: {bad}"
        assert g["root"].hex() == o["root"], f"config {cfg} layer {li}: witness root"
        z = hashlib.sha256(np.ascontiguousarray(g["Z"].cpu().numpy().astype("<i8")).tobytes()).hexdigest()
        assert z == ofp["digests"]["Z"] == o["digests"]["Z"]
    torch.cuda.synchronize()
