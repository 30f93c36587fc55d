"""The C-ABI library on the host: it loads, exports every symbol that
include/ra.h declares, rejects bad arguments before touching a device, and
its host-only verifier (ra_verify) accepts the oracle's honest transcripts
and rejects tampered ones.  No GPU compute call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

from helpers import oracle_layer_for_abi
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def ra():
    from paper_2505_17623_amd import ra as ra_mod
    if not os.path.exists(ra_mod.LIB_PATH):
        from paper_2505_17623_amd import build
        build.build()
    ra_mod.lib()
    return ra_mod


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "ra.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ra_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(ra):
    syms = declared_symbols()
    assert set(syms) == set(ra.EXPORTS), syms
    L = ctypes.CDLL(ra.LIB_PATH)
    for s in syms:
        assert hasattr(L, s), s


def test_commit_batch_workspace_size(ra):
    """ra_commit_batch_workspace_size: one table's region per table (each as
    ra_commit's, rounded to 256 bytes) plus 64 output bytes per table; no
    tables or an unknown type is RA_E_INVAL, more than 64 tables
    RA_E_NOT_IMPLEMENTED."""
    L = ra.lib()
    types = [ra.RA_I16, ra.RA_U16, ra.RA_I32, ra.RA_U64]
    single = []
    for t in types:
        sz = ctypes.c_size_t()
        assert L.ra_commit_workspace_size(t, ctypes.byref(sz)) == 0
        single.append(sz.value - 256)  # ra_commit's region: the tables' sums, then 256 bytes of output
    dts = (ctypes.c_int32 * 4)(*types)
    sz = ctypes.c_size_t()
    assert L.ra_commit_batch_workspace_size(dts, 4, ctypes.byref(sz)) == 0
    assert sz.value == sum((b + 255) // 256 * 256 for b in single) + 64 * 4 + 256
    assert L.ra_commit_batch_workspace_size(dts, 0, ctypes.byref(sz)) == -1
    many = (ctypes.c_int32 * 65)(*([ra.RA_I32] * 65))
    assert L.ra_commit_batch_workspace_size(many, 65, ctypes.byref(sz)) == -9
    bad = (ctypes.c_int32 * 2)(ra.RA_I32, ra.RA_I64)
    assert L.ra_commit_batch_workspace_size(bad, 2, ctypes.byref(sz)) == -1


def test_host_side_argument_errors(ra):
    L = ra.lib()
    h = ctypes.c_void_p()
    assert L.ra_ctx_create(7, 1, None, ctypes.byref(h)) == -2                     # unsupported prime
    assert L.ra_ctx_create(ra.P61, 1, None, None) == -1                           # null out
    assert L.ra_ctx_create(ra.P61, 0, None, ctypes.byref(h)) == -5                # seed 0
    assert L.ra_ctx_create_stream(7, None, 0, None, ctypes.byref(h)) == -2
    bad = np.array([ra.P61], dtype=np.uint64)
    assert L.ra_ctx_create_stream(ra.P61, bad.ctypes.data_as(ra.u64p), 1, None, ctypes.byref(h)) == -5
    assert L.ra_ctx_destroy(None) == -1
    for code, name in ra.STATUS.items():
        assert L.ra_status_str(code)
    v = ctypes.c_int32()
    f = ctypes.c_uint32()
    assert L.ra_verify_stream(ra.P61, None, 0, 0, None, None, None, ctypes.byref(v), ctypes.byref(f)) == 0
    assert L.ra_verify_stream(5, None, 0, 0, None, None, None, ctypes.byref(v), ctypes.byref(f)) == -2
    assert L.ra_verify(ra.P61, 1, 0, None, None, None, ctypes.byref(v), ctypes.byref(f)) == 0
    assert L.ra_verify(ra.P61, 0, 0, None, None, None, ctypes.byref(v), ctypes.byref(f)) == -5
    assert L.ra_verify(5, 1, 0, None, None, None, ctypes.byref(v), ctypes.byref(f)) == -2
    # workspace size: powers of two only; this GPU path's limits
    sz = ctypes.c_size_t()
    assert L.ra_workspace_size(3, 4, 4, 64, ctypes.byref(sz)) == -1
    assert L.ra_workspace_size(4, 4, 4, 48, ctypes.byref(sz)) == -1
    assert L.ra_workspace_size(4, 1 << 16, 4, 64, ctypes.byref(sz)) == -9          # m > 32768
    assert L.ra_workspace_size(1 << 16, 4, 1 << 16, 64, ctypes.byref(sz)) == -9    # N > 2^31
    assert L.ra_workspace_size(4, 4, 4, 128, ctypes.byref(sz)) == -9               # P > 64
    # the fixed-scratch binding rejects before touching a device: a table whose
    # eq table (2^20 words) exceeds the scratch, a bad dimension, a bad point
    fake = ctypes.c_void_p(1 << 20)
    pt = np.zeros(20, dtype=np.uint64)
    assert L.ra_mle_bind_noalloc(fake, ra.RA_I16, 1 << 20, 1, 1, pt.ctypes.data_as(ra.u64p), 20, fake,
                                 None) == -10
    assert L.ra_mle_bind_noalloc(fake, ra.RA_I16, 3, 4, 1, pt.ctypes.data_as(ra.u64p), 2, fake, None) == -1
    assert L.ra_mle_bind_noalloc(fake, ra.RA_I16, 4, 4, 1, pt.ctypes.data_as(ra.u64p), 3, fake, None) == -1
    big = np.array([ra.P61, 0], dtype=np.uint64)
    assert L.ra_mle_bind_noalloc(fake, ra.RA_I16, 4, 4, 1, big.ctypes.data_as(ra.u64p), 2, fake, None) == -1


def oracle_network(wl):
    outs = orc.prove_network(wl)
    layers = []
    for li, res in enumerate(outs):
        layers.append(oracle_layer_for_abi(res, wl.layers[li].B, chained=li > 0 and wl.links[li] is None))
    return layers


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_library_verifier_accepts_oracle_transcripts(ra, cfg):
    wl = inputs.small(cfg)
    layers = oracle_network(wl)
    assert ra.ra_verify(wl.challenges, layers) == (0, 0)
    # the seeded form draws the stream with the library's own generator: it
    # accepts only if that stream equals the one the oracle was given
    assert ra.ra_verify(wl.challenge_seed, layers) == (0, 0)
    assert ra.ra_verify(wl.challenge_seed + 1, layers)[0] != 0


def test_workspace_size_covers_layers(ra):
    small = ra.workspace_size(64, 64, 64, 64)
    big = ra.workspace_size(1024, 1024, 1024, 64)
    assert 0 < small < big
    # the range call's tables (three of N words with ReLU) bound it below
    assert big >= 3 * 8 * 1024 * 1024


def test_library_verifier_rejects_tampering(ra):
    wl = inputs.small(2)
    base = oracle_network(wl)

    def check(li, mutate):
        layers = [dict(L, transcript=dict(L["transcript"])) for L in base]
        layers[li] = dict(layers[li])
        mutate(layers[li])
        v, f = ra.ra_verify(wl.challenges, layers)
        assert v != 0 and f == li
        return v

    P = ra.P61

    def bump(key, i=None):
        def f(L):
            tr = L["transcript"]
            if i is None:
                tr[key] = (tr[key] + 1) % P
            else:
                ev = list(tr[key]); ev[i] = (ev[i] + 1) % P; tr[key] = ev
        return f

    for key in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim", "bits_claim",
                "range_sum"):
        check(0, bump(key))
    for key in ("mm_evals", "rs_evals", "zc_evals"):
        check(1, bump(key, 0))
        check(1, bump(key, -1))

    def flip_bit(L):
        b = L["bits"].copy(); b[3] ^= np.uint64(1 << 2); L["bits"] = b
    assert check(0, flip_bit) == 7

    def wrong_output(L):
        Z = L["Z"].copy(); Z.flat[5] += 1; L["Z"] = Z
    assert check(2, wrong_output) == 11

    def relu_sign(L):
        R = L["R"]; idx = int(np.argmax(R.reshape(-1) < 0))
        Y = L["Y"].copy(); Y.flat[idx] = R.flat[idx]; L["Y"] = Y
    assert check(0, relu_sign) != 0

    def unchained(L):
        A = L["A"].copy(); A.flat[0] += 1; L["A"] = A
    assert check(1, unchained) == 14


def test_library_verifier_openings(ra):
    """Tampers that keep every identity before an opening true (a* b* and
    r_at^2 - y_at^2 unchanged, or a public matrix entry changed), so only
    the openings of the final claims against the tables (check 3: a*, b*
    against A, B; check 10: r_at, y_at against R, Y) can reject them."""
    wl = inputs.small(2)
    base = oracle_network(wl)
    P = ra.P61
    inv2 = pow(2, P - 2, P)

    def verdict(li, **over):
        layers = [dict(L, transcript=dict(L["transcript"])) for L in base]
        for key, val in over.items():
            if key in ("A", "B"):
                layers[li][key] = val
            else:
                layers[li]["transcript"][key] = val
        return ra.ra_verify(wl.challenges, layers)

    tr0 = base[0]["transcript"]
    assert verdict(0, a_star=2 * tr0["a_star"] % P, b_star=tr0["b_star"] * inv2 % P) == (3, 0)
    assert verdict(0, r_at=(P - tr0["r_at"]) % P) == (10, 0)
    assert verdict(0, y_at=(P - tr0["y_at"]) % P) == (10, 0)
    A = base[0]["A"].copy(); A.flat[7] += 1
    assert verdict(0, A=A) == (3, 0)
    B = base[1]["B"].copy(); B.flat[3] -= 1
    assert verdict(1, B=B) == (3, 1)


def linked_network(wl):
    """The oracle's proof of a workload with its gather links, as ra_verify's layers."""
    outs = orc.prove_network(wl, links=True)
    layers = []
    for li, res in enumerate(outs):
        L = oracle_layer_for_abi(res, wl.layers[li].B, chained=li > 0 and wl.links[li] is None)
        if "link" in res:
            L["link_src"] = wl.link_map(li).astype(np.int32)
            L["link"] = res["link"]
        layers.append(L)
    return layers


def test_library_verifier_gather_links(ra):
    """ra_verify on the oracle's proof of the small CNN with its im2col and
    flatten links: accepted (stream and seed), and each link tamper rejected
    with verdict 15 at its layer."""
    wl = inputs.small(4)
    base = linked_network(wl)
    assert sum("link" in L for L in base) == len(base) - 1
    assert ra.ra_verify(wl.challenges, base) == (0, 0)
    assert ra.ra_verify(wl.challenge_seed, base) == (0, 0)
    P = ra.P61
    half = (P + 1) // 2

    def verdict(li, **over):
        layers = [dict(L) for L in base]
        layers[li] = dict(layers[li], **over)
        return ra.ra_verify(wl.challenges, layers)

    for li in (1, 3, 4):
        lk = base[li]["link"]
        ev = list(lk["evals"])
        ev[0] = (ev[0] + 1) % P
        assert verdict(li, link=dict(lk, evals=ev)) == (15, li)
        ev = list(lk["evals"])
        ev[-1] = (ev[-1] + 1) % P
        assert verdict(li, link=dict(lk, evals=ev)) == (15, li)
        # the final product kept: only the opening of Z_prev at y* fails
        assert verdict(li, link=dict(lk, z_at=2 * lk["z_at"] % P, w_at=lk["w_at"] * half % P)) == (15, li)
        src = base[li]["link_src"].copy()
        j = int(np.flatnonzero(src >= 0)[0])
        src[j] = (src[j] + 1) % (base[li - 1]["Z"].size)
        assert verdict(li, link_src=src) == (15, li)                  # another public map: W~ fails
        src = base[li]["link_src"].copy()
        src[0] = base[li - 1]["Z"].size                               # outside the previous output
        assert verdict(li, link_src=src) == (15, li)
        assert verdict(li, link=dict(lk, evals=lk["evals"][:-3])) == (15, li)
    # with a link, A itself is not opened: a* is tied to Z_prev by the link
    A = base[2]["A"].copy()
    A.flat[5] += 1
    assert verdict(2, A=A) == (0, 0)
    # a changed previous output breaks that layer's own openings first
    Z = base[1]["Z"].copy()
    Z.flat[0] += 1
    assert verdict(1, Z=Z)[0] != 0


def test_link_host_side_errors(ra):
    L = ra.lib()
    sz = ctypes.c_size_t()
    assert L.ra_link_workspace_size(3, 4, 4, ctypes.byref(sz)) == -1
    assert L.ra_link_workspace_size(4, 3, 4, ctypes.byref(sz)) == -1
    assert L.ra_link_workspace_size(1 << 32, 4, 4, ctypes.byref(sz)) == -9
    assert L.ra_link_workspace_size(1 << 20, 4, 4, ctypes.byref(sz)) == 0 and sz.value >= 8 << 20
    pr = ra.LinkProof()
    assert L.ra_link_prove(None, None, 4, None, 4, None, 0, ctypes.byref(pr)) == -1


def fs_layers(wl, res):
    from helpers import pack_planes
    layers = []
    for li, r in enumerate(res):
        chained = li > 0 and wl.links[li] is None
        A = np.ascontiguousarray(r["A"], dtype=np.int32 if chained or np.abs(r["A"]).max() >= 2 ** 15 else np.int16)
        layers.append(dict(A=A, B=wl.layers[li].B, Z=r["Z"].astype(np.int32), R=r["R"].astype(np.int32),
                           Rm=r["Rm"].astype(np.uint16), Y=r["Y"].astype(np.int32), bits=pack_planes(r["bits"]),
                           transcript=r, chained=chained))
    return layers


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_library_fs_verifier_on_oracle_proofs(ra, cfg):
    """ra_verify_fs replays the oracle's non-interactive proofs: accepted;
    another domain, public digest, round word or witness entry rejected, with
    the verdict the oracle's own verifier gives."""
    import hashlib
    wl = inputs.small(cfg)
    domain = hashlib.sha256(wl.name.encode()).digest()
    pubs = [hashlib.sha256(f"{wl.name}/layer {li}".encode()).digest() for li in range(len(wl.layers))]
    res = orc.prove_network_fs(wl, domain, pubs)
    layers = fs_layers(wl, res)
    assert ra.ra_verify_fs(domain, pubs, layers) == (0, 0)
    assert ra.ra_verify_fs(hashlib.sha256(b"x").digest(), pubs, layers)[0] != 0
    assert ra.ra_verify_fs(domain, [bytes(32)] + pubs[1:], layers)[0] != 0
    last = len(layers) - 1

    def both(changed_tr=None, **tables):
        L = [dict(x) for x in layers]
        if changed_tr is not None:
            L[last]["transcript"] = changed_tr
        L[last].update(tables)
        got = ra.ra_verify_fs(domain, pubs, L)
        st = orc.fs_init(domain)
        v = 0
        for li, x in enumerate(L):
            tr = x["transcript"]
            planes = ra.unpack_bits(x["bits"], tr["P"]).astype(np.int64)
            v = orc.verify_layer_fs(x["A"], x["B"], x["Z"], tr["s"], tr["relu"], tr["mode"], x["R"],
                                    x["Rm"], x["Y"], planes, tr, st, pubs[li])
            if v:
                break
        return got, v

    r = res[last]
    ev = list(r["rs_evals"])
    ev[3] = ((ev[3][0] + 1) % ra.P61, ev[3][1])
    (v, li), ov = both(dict(r, rs_evals=ev))
    assert v != 0 and li == last and v == ov
    (v, li), ov = both(dict(r, a_star=(r["a_star"][0], (r["a_star"][1] + 5) % ra.P61)))
    assert v != 0 and li == last and v == ov
    R = layers[last]["R"].copy()
    R.flat[0] += 1
    (v, li), ov = both(R=R)
    assert v != 0 and li == last and v == ov


@pytest.mark.parametrize("dtype", [np.int16, np.uint16, np.int32, np.uint64])
def test_library_commitment_opening_matches_oracle(ra, dtype):
    """ra_commit_open (the library's secp256k1 arithmetic, run on the host)
    accepts the oracle's commitment to the same values and generators and
    rejects another value vector or another point."""
    import hashlib
    from oracle import ec_oracle as ec
    domain = hashlib.sha256(b"commit abi").digest()
    gens = ec.generators(domain, 12)
    limbs = ra.point_limbs(gens)
    rng = np.random.default_rng(4)
    info = np.iinfo(dtype)
    v = rng.integers(info.min, info.max, size=12, dtype=dtype, endpoint=True)
    v[0] = info.min
    v[1] = info.max
    v[2] = 0
    P = ec.encode(ec.commit([int(x) for x in v], gens))
    assert ra.commit_open(v, limbs, P)
    w = v.copy()
    w[5] = w[5] ^ 1
    assert not ra.commit_open(w, limbs, P)
    assert not ra.commit_open(v, limbs, ec.encode(ec.add(ec.decode(P), gens[0])))
    assert ra.commit_open(np.zeros(12, dtype=dtype), limbs, bytes(64))


def test_commitment_field_product_top_limb(ra):
    """A product whose high half is within 2^-22 of 2^256 leaves more than 32
    bits above 2^256 after the first reduction: doubling the curve point with
    x = q - 3 squares q - 3, which does.  The host opening (the same limb code
    as the device) must agree with the oracle there."""
    from oracle import ec_oracle as ec
    x = ec.Q - 3
    rhs = (pow(x, 3, ec.Q) + 7) % ec.Q
    y = pow(rhs, (ec.Q + 1) // 4, ec.Q)
    P = (x, y)
    assert ec.on_curve(P)
    limbs = ra.point_limbs([P, ec.G])
    for vals in ([2, 0], [3, 0], [-5, 7], [2 ** 31 - 1, -(2 ** 31)]):
        want = ec.encode(ec.commit(vals, [P, ec.G]))
        assert ra.commit_open(np.array(vals, dtype=np.int32), limbs, want), vals
