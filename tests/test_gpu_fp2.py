"""The GPU prover over F_{p^2} = F_p[i] / (i^2 + 1) (ra_prove_layer_fp2)
against the F_{p^2} oracle, through the C ABI.

Every transcript word (each a pair re, im) and every output table must be
bit-identical.  Small workloads and edge shapes compare element by element;
the full workloads compare with the oracle's transcripts stored in
tests/golden/full_fp2_cfg<N>.json (written by make_golden.py --fp2, which
calls only the oracle) and with the table digests of tests/golden/full_cfg<N>.json
(the witness does not depend on the field of the challenges).
"""
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


def diff_fp2(tr, want):
    return [k for k in KEYS if as_pairs(tr[k]) != as_pairs(want[k])]


def compare_layer(ra, g, o, label):
    tr = g["transcript"]
    bad = diff_fp2(tr, o)
    assert not bad, f"{label}: transcript words differ in {bad}"
    assert np.array_equal(g["C"].cpu().numpy(), o["C"]), label
    for key in ("R", "Y", "Z"):
        assert np.array_equal(g[key].cpu().numpy().astype(np.int64), o[key]), (label, key)
    assert np.array_equal(g["Rm"].cpu().numpy().view(np.uint16).astype(np.int64), o["Rm"]), label
    assert np.array_equal(ra.unpack_bits(g["bits"].cpu().numpy(), tr["P"]), o["bits"]), label


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("source", ["array", "seed"])
def test_fp2_network_parity_small(ra, cfg, source):
    wl = inputs.small(cfg)
    want = orc.prove_network_fp2(wl)
    ctx = ra.Context(orc.fp2_stream(wl)) if source == "array" else ra.Context(seed=wl.challenge_seed)
    got = ra.prove_network_fp2(ctx, wl)
    for li, (g, o) in enumerate(zip(got, want)):
        assert np.array_equal(g["A"].cpu().numpy(), o["A"]), f"cfg{cfg} L{li} input"
        compare_layer(ra, g, o, f"cfg{cfg} L{li}")
    assert ctx.cursor() == want[-1]["cursor"]


# (n, m, k, s, relu, mode, |entries| bound)
SHAPES = [
    (1, 1, 1, 3, True, 0, 3000),        # every sum-check instance degenerate (no matrix or ReLU rounds)
    (1, 8, 1, 4, False, 0, 3000),
    (2, 1, 4, 2, True, 1, 3000),
    (8, 16384, 1, 9, True, 0, 64),      # long matrix instance, N = 8
    (1, 4, 16384, 5, False, 1, 3000),   # range instance over 2^14 entries
    (128, 64, 128, 11, True, 0, 3000),  # several blocks in the first rounds of every instance
    (32, 32, 64, 6, True, 1, 3000),
    (256, 8, 512, 12, True, 1, 3000),   # 2^17 entries: the first rounds run on the block limit
]


@pytest.mark.parametrize("n,m,k,s,relu,mode,mag", SHAPES)
def test_fp2_layer_parity_shapes(ra, n, m, k, s, relu, mode, mag):
    rng = np.random.default_rng(n * 131 + m * 7 + k)
    A = rng.integers(-mag, mag, size=(n, m)).astype(np.int16)
    B = rng.integers(-mag, mag, size=(m, k)).astype(np.int16)
    chal = inputs.xorshift64_stream(99 + n + m + k, 1024)
    o = orc.prove_layer_fp2(A, B, s, relu, mode, chal)
    ctx = ra.Context(chal)
    g = ra.prove_layer_fp2(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), s, relu, mode)
    compare_layer(ra, g, o, f"{n}x{m}x{k}")
    assert ctx.cursor() == o["cursor"]


def test_fp2_int32_input_and_given_t(ra):
    rng = np.random.default_rng(3)
    A = rng.integers(-(2 ** 16), 2 ** 16, size=(32, 64)).astype(np.int32)
    B = rng.integers(-(2 ** 10), 2 ** 10, size=(64, 16)).astype(np.int16)
    chal = inputs.xorshift64_stream(1234, 1024)
    o = orc.prove_layer_fp2(A, B, 12, True, 0, chal, t_in=-1)
    t_big = o["t"] + 2
    o2 = orc.prove_layer_fp2(A, B, 12, True, 0, chal, t_in=t_big)
    for want, t in ((o, -1), (o2, t_big)):
        ctx = ra.Context(chal)
        g = ra.prove_layer_fp2(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), 12, True, 0, t)
        compare_layer(ra, g, want, f"t={t}")


def test_fp2_errors(ra):
    chal = inputs.xorshift64_stream(77, 256)
    A = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    B = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    with pytest.raises(ra.RAError) as e:                       # a given t that R does not fit
        ra.prove_layer_fp2(ra.Context(chal), A, B, 4, True, 0, t=3)
    assert e.value.code == -4
    with pytest.raises(ra.RAError) as e:                       # too few challenges
        ra.prove_layer_fp2(ra.Context(chal[:5]), A, B, 4, True, 0)
    assert e.value.code == -5
    with pytest.raises(ra.RAError) as e:                       # non power of two
        ra.prove_layer_fp2(ra.Context(chal), A[:3].contiguous(), B, 4, True, 0)
    assert e.value.code == -1


def layers_for_verifier(ra, wl, got):
    return [dict(A=g["A"].cpu().numpy(), B=wl.layers[li].B, Z=g["Z"].cpu().numpy(), R=g["R"].cpu().numpy(),
                 Rm=g["Rm"].cpu().numpy(), Y=g["Y"].cpu().numpy(), bits=g["bits"].cpu().numpy(),
                 transcript=g["transcript"], chained=li > 0) for li, g in enumerate(got)]


@pytest.mark.parametrize("cfg", [2, 5])
def test_fp2_transcripts_verify_both_ways(ra, cfg):
    """The GPU's F_{p^2} proofs pass the oracle's verifier and the library's;
    a changed word in any part of the transcript is rejected by both."""
    wl = inputs.small(cfg)
    chal = orc.fp2_stream(wl)
    got = ra.prove_network_fp2(ra.Context(seed=wl.challenge_seed), wl)
    layers = layers_for_verifier(ra, wl, got)
    cur = 0
    for L in layers:
        tr = L["transcript"]
        planes = ra.unpack_bits(L["bits"], tr["P"]).astype(np.int64)
        v, cur = orc.verify_layer_fp2(L["A"], L["B"], L["Z"], tr["s"], tr["relu"], tr["mode"], L["R"],
                                      L["Rm"].view(np.uint16), L["Y"], planes, tr, chal, cur)
        assert v == 0
    assert ra.ra_verify_fp2(wl.challenge_seed, layers) == (0, 0)
    last = 0                                 # a layer with ReLU: r_at and y_at are read only there
    assert wl.layers[last].relu
    for key, idx in (("c0", None), ("mm_evals", 0), ("rs_evals", -1), ("bits_claim", None), ("y_at", None),
                     ("zc_evals", 1)):
        orig = layers[last]["transcript"]
        if idx is None:
            re, im = orig[key]
            changed = dict(orig, **{key: (re, (im + 1) % P61)})
        else:
            ev = list(orig[key])
            if not ev:
                continue
            re, im = ev[idx]
            ev[idx] = ((re + 1) % P61, im)
            changed = dict(orig, **{key: ev})
        layers[last]["transcript"] = changed
        verdict, failed = ra.ra_verify_fp2(wl.challenge_seed, layers)
        assert verdict != 0 and failed == last, key
        L = layers[last]
        planes = ra.unpack_bits(L["bits"], changed["P"]).astype(np.int64)
        v, _ = orc.verify_layer_fp2(L["A"], L["B"], L["Z"], changed["s"], changed["relu"], changed["mode"], L["R"],
                                    L["Rm"].view(np.uint16), L["Y"], planes, changed, chal, 0)
        assert v == verdict, key
        layers[last]["transcript"] = orig


def digest_i64(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(np.asarray(a).astype("<i8")).tobytes()).hexdigest()


def digest(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_fp2_full_workload_matches_oracle(ra, cfg):
    """Full size, in the launch configuration of the F_{p^2} bench line: a
    context drawing its stream from the seed, deferred, t given, buffers kept."""
    path = os.path.join(GOLD, f"full_fp2_cfg{cfg}.json")
    gold = json.load(open(path))
    gold_fp = json.load(open(os.path.join(GOLD, f"full_cfg{cfg}.json")))
    wl = inputs.workload(cfg, "full")
    ctx = ra.Context(seed=wl.challenge_seed, deferred=True)
    got = ra.prove_network_fp2(ctx, wl, ts=[o["transcript"]["t"] for o in gold["layers"]], bufs=[])
    ctx.sync()
    used = 0
    for li, (g, o, ofp) in enumerate(zip(got, gold["layers"], gold_fp["layers"])):
        bad = diff_fp2(g["transcript"], o["transcript"])
        assert not bad, f"config {cfg} layer {li}: transcript words differ in {bad}"
        used += o["transcript"]["challenges_used"]
        d = ofp["digests"]
        assert digest_i64(g["A"].cpu().numpy()) == d["A"], f"config {cfg} layer {li}: input A"
        assert digest_i64(g["C"].cpu().numpy()) == d["C"], f"config {cfg} layer {li}: C"
        for key in ("R", "Y", "Z"):
            assert digest_i64(g[key].cpu().numpy()) == d[key], f"config {cfg} layer {li}: {key}"
        assert digest_i64(g["Rm"].cpu().numpy().view(np.uint16)) == d["Rm"], f"config {cfg} layer {li}: Rm"
        planes = ra.unpack_bits(g["bits"].cpu().numpy(), g["transcript"]["P"])
        assert digest(planes) == d["bits"], f"config {cfg} layer {li}: bit planes"
        assert o["digests"]["Z"] == d["Z"]
        del planes
    assert ctx.cursor() == used
    torch.cuda.synchronize()
