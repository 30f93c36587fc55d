"""GPU prover vs the CPU oracle, element by element, through the C ABI.

Every transcript word (round polynomials, claims, final values, t, P) and
every output table (C, R, Rm, Y, Z, the bit planes) must be bit-identical.
Sizes are ones the oracle finishes in seconds while spanning several tiles
and the global-round / LDS-tail boundary of every sum-check instance.
"""
import numpy as np
import pytest
import torch

from helpers import diff_transcripts, oracle_layer_for_abi
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

pytestmark = pytest.mark.gpu
P61 = (1 << 61) - 1


@pytest.fixture(scope="module")
def ra():
    from paper_2505_17623_amd import ra as ra_mod
    ra_mod.lib()
    assert torch.cuda.is_available()
    return ra_mod


def compare_layer(ra, g, o, label=""):
    tr = g["transcript"]
    bad = diff_transcripts(tr, o)
    assert not bad, f"{label}: transcript mismatch in {bad}"
    assert np.array_equal(g["C"].cpu().numpy(), o["C"]), label
    for key in ("R", "Y", "Z"):
        assert np.array_equal(g[key].cpu().numpy().astype(np.int64), o[key]), (label, key)
    assert np.array_equal(g["Rm"].cpu().numpy().view(np.uint16).astype(np.int64), o["Rm"]), label
    planes = ra.unpack_bits(g["bits"].cpu().numpy(), tr["P"])
    assert np.array_equal(planes, o["bits"]), label
    words = g["bits"].cpu().numpy().view(np.uint64)
    assert not np.any(words >> np.uint64(tr["P"])) if tr["P"] < 64 else True


# --- multilinear binding -----------------------------------------------------
EDGE = {np.int16: [-32768, 32767, -1, 0, 1], np.int32: [-(2 ** 31), 2 ** 31 - 1, -1, 0, 1],
        np.int64: [-(2 ** 62), 2 ** 62, -1, 0, (1 << 61) - 1, -((1 << 61) - 1)]}


@pytest.mark.parametrize("shape", [(1, 1), (4, 8), (64, 32), (512, 256), (8, 2048), (128, 1)])
@pytest.mark.parametrize("dt", [np.int16, np.int32, np.int64, "field"])
def test_mle_bind_parity(ra, shape, dt):
    rows, cols = shape
    rng = np.random.default_rng(rows * 7 + cols)
    if dt == "field":
        T = rng.integers(0, P61, size=shape, dtype=np.uint64)
        T.flat[0] = P61 - 1
        host = T.astype(object)
        dev = torch.from_numpy(T.view(np.int64)).cuda()
    else:
        info = np.iinfo(dt)
        T = rng.integers(info.min, info.max, size=shape, dtype=dt, endpoint=True)
        if dt == np.int64:
            T = rng.integers(-(2 ** 62), 2 ** 62, size=shape, dtype=np.int64)
        for i, e in enumerate(EDGE[dt][:T.size]):
            T.flat[i] = e
        host = T.astype(object)
        dev = torch.from_numpy(T).cuda()
    ctx = ra.Context(inputs.xorshift64_stream(5, 8))
    for bind_rows in (True, False):
        v = (rows if bind_rows else cols).bit_length() - 1
        z = [int(x) for x in inputs.xorshift64_stream(11 + v + bind_rows, max(v, 1))[:v]]
        out = ra.ra_mle_bind(ctx, dev, bind_rows, z, field=(dt == "field")).cpu().numpy().view(np.uint64)
        if bind_rows:
            want = [orc.mle_field([int(x) % P61 for x in host[:, c]], z) for c in range(cols)]
        else:
            want = [orc.mle_field([int(x) % P61 for x in host[r, :]], z) for r in range(rows)]
        assert [int(x) for x in out] == want


# --- whole layers and networks ----------------------------------------------
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_network_parity_small(ra, cfg):
    wl = inputs.small(cfg)
    want = orc.prove_network(wl)
    ctx = ra.Context(wl.challenges)
    got = ra.prove_network(ctx, wl)
    for li, (g, o) in enumerate(zip(got, want)):
        assert np.array_equal(g["A"].cpu().numpy(), o["A"]), f"cfg{cfg} L{li} input"
        compare_layer(ra, g, o, f"cfg{cfg} L{li}")
    assert ctx.cursor() == want[-1]["cursor"]


# (n, m, k, s, relu, mode, |entries| bound): keeps s + (t + 2)(1 + relu) <= 64
SHAPES = [
    (1, 1, 1, 3, True, 0, 3000),
    (1, 8, 1, 4, False, 0, 3000),
    (2, 1, 4, 2, True, 1, 3000),
    (8, 16384, 1, 9, True, 0, 64),      # m beyond the matrix instance's LDS tail -> global rounds
    (1, 4, 16384, 5, False, 1, 3000),   # N beyond the range instance's LDS tail
    (128, 64, 128, 11, True, 0, 3000),  # N beyond the ReLU instance's LDS tail, several GEMM tiles
    (32, 32, 64, 6, True, 1, 3000),
    (1, 64, 8, 7, True, 0, 3000),       # fused front: one row, the narrowest B it takes
    (2048, 64, 8, 10, True, 0, 3000),   # fused front: eight row chunks of A accumulated
    (64, 2048, 16, 10, False, 1, 3000), # fused front feeding a global round (m beyond the LDS tail)
    (4, 4096, 8, 8, True, 0, 3000),     # two global rounds reading the fused front's accumulators
    (2, 8192, 8, 9, False, 1, 3000),    # three global rounds
    (16, 4096, 1024, 10, True, 0, 3000),  # fused front with four rows per column-binding wave (its longest-first
                                          # role order) and two column steps per row
]


@pytest.mark.parametrize("n,m,k,s,relu,mode,mag", SHAPES)
def test_layer_parity_shapes(ra, n, m, k, s, relu, mode, mag):
    rng = np.random.default_rng(n * 131 + m * 7 + k)
    A = rng.integers(-mag, mag, size=(n, m)).astype(np.int16)
    B = rng.integers(-mag, mag, size=(m, k)).astype(np.int16)
    chal = inputs.xorshift64_stream(99 + n + m + k, 512)
    o = orc.prove_layer(A, B, s, relu, mode, chal)
    ctx = ra.Context(chal)
    g = ra.prove_layer(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), s, relu, mode)
    compare_layer(ra, g, o, f"{n}x{m}x{k}")


def test_int32_input_and_given_t(ra):
    rng = np.random.default_rng(3)
    A = rng.integers(-(2 ** 16), 2 ** 16, size=(32, 64)).astype(np.int32)
    B = rng.integers(-(2 ** 10), 2 ** 10, size=(64, 16)).astype(np.int16)
    chal = inputs.xorshift64_stream(1234, 512)
    o = orc.prove_layer(A, B, 12, True, 0, chal, t_in=-1)
    t_big = o["t"] + 2
    o2 = orc.prove_layer(A, B, 12, True, 0, chal, t_in=t_big)
    for want, t in ((o, -1), (o2, t_big)):
        ctx = ra.Context(chal)
        g = ra.prove_layer(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), 12, True, 0, t)
        compare_layer(ra, g, want, f"t={t}")


def test_errors_and_state(ra):
    chal = inputs.xorshift64_stream(77, 256)
    A = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    B = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    ctx = ra.Context(chal)
    C, _ = ra.ra_sumcheck_matmul_prove(ctx, A, B)
    with pytest.raises(ra.RAError) as e:                     # a given t that R does not fit
        ra.ra_rescale_relu_witness(ctx, C, 4, True, 0, t=3)
    assert e.value.code == -4
    with pytest.raises(ra.RAError) as e:                     # matmul again before the witness
        ra.ra_sumcheck_matmul_prove(ctx, A, B)
    assert e.value.code == -7
    (R, Rm, Y, Z, bits), info = ra.ra_rescale_relu_witness(ctx, C, 4, True, 0)
    assert info.t >= 0
    ra.ra_range_prove(ctx, bits, R, Y, info)
    short = ra.Context(chal[:3])
    with pytest.raises(ra.RAError) as e:
        ra.ra_sumcheck_matmul_prove(short, A, B)
    assert e.value.code == -5
    with pytest.raises(ra.RAError) as e:                     # non power of two
        ra.ra_sumcheck_matmul_prove(ra.Context(chal), A[:3].contiguous(), B)
    assert e.value.code == -1


def test_gpu_transcripts_verify_both_ways(ra):
    wl = inputs.small(2)
    ctx = ra.Context(wl.challenges)
    got = ra.prove_network(ctx, wl)
    layers = []
    cur = 0
    for li, g in enumerate(got):
        L = dict(A=g["A"].cpu().numpy(), B=wl.layers[li].B, Z=g["Z"].cpu().numpy(), R=g["R"].cpu().numpy(),
                 Rm=g["Rm"].cpu().numpy(), Y=g["Y"].cpu().numpy(), bits=g["bits"].cpu().numpy(),
                 transcript=g["transcript"], chained=li > 0)
        layers.append(L)
        tr = dict(g["transcript"])
        planes = ra.unpack_bits(L["bits"], tr["P"]).astype(np.int64)
        v, cur = orc.verify_layer(L["A"], L["B"], L["Z"], tr["s"], tr["relu"], tr["mode"], L["R"],
                                  L["Rm"].view(np.uint16), L["Y"], planes, tr, wl.challenges, cur)
        assert v == 0, li
    assert ra.ra_verify(wl.challenges, layers) == (0, 0)
    layers[1]["transcript"] = dict(layers[1]["transcript"], bits_claim=(layers[1]["transcript"]["bits_claim"] + 1) % P61)
    assert ra.ra_verify(wl.challenges, layers)[0] != 0


@pytest.mark.parametrize("a_dtype,n,m,k", [(np.int16, 64, 128, 64), (np.int32, 32, 256, 128),
                                           (np.int32, 1, 64, 1), (np.int16, 128, 32768, 2)])
def test_matmul_extreme_values(ra, a_dtype, n, m, k):
    """Exact product and matrix sum-check at the edges of the limb split:
    int32 inputs near +-2^31, int16 at -32768 / 32767, the largest inner
    dimension (2^15), and tiles that are not full."""
    rng = np.random.default_rng(n + m + k)
    info = np.iinfo(a_dtype)
    A = rng.integers(info.min, info.max, size=(n, m), dtype=np.int64, endpoint=True).astype(a_dtype)
    B = rng.integers(-32768, 32767, size=(m, k), dtype=np.int64, endpoint=True).astype(np.int16)
    A.flat[:4] = [info.min, info.max, -1, 0][:A.size]
    B.flat[:4] = [-32768, 32767, -1, 0][:B.size]
    if m == 32768:                      # worst case for the int32 limb accumulators
        A[:, :] = info.min
        B[:, 0] = -32768
    chal = inputs.xorshift64_stream(555 + m, 512)
    o = orc.prove_layer(A, B, 30, False, 0, chal)  # s = 30 keeps the oracle's t small; only C and the
    ctx = ra.Context(chal)                          # matrix transcript are compared
    C, mm = ra.ra_sumcheck_matmul_prove(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
    want = (A.astype(object) @ B.astype(object))
    assert np.array_equal(C.cpu().numpy().astype(object), want)
    assert np.array_equal(C.cpu().numpy(), o["C"])
    for key in ("c0", "mm_evals", "a_star", "b_star"):
        assert mm[key] == o[key], key


@pytest.mark.parametrize("a_dtype,n,m,k", [(np.int16, 4096, 128, 512), (np.int32, 4096, 64, 512),
                                           (np.int32, 8192, 256, 64)])
def test_product_many_tiles(ra, a_dtype, n, m, k):
    """Products with more output tiles than compute units, at the edges of
    the limb split; C against the exact integer product."""
    rng = np.random.default_rng(n + m + k + 1)
    info = np.iinfo(a_dtype)
    A = rng.integers(info.min, info.max, size=(n, m), dtype=np.int64, endpoint=True).astype(a_dtype)
    B = rng.integers(-32768, 32767, size=(m, k), dtype=np.int64, endpoint=True).astype(np.int16)
    A[0, :] = info.min
    B[:, 0] = -32768
    A[1, :] = info.max
    B[:, 1] = 32767
    chal = inputs.xorshift64_stream(999 + n, 512)
    ctx = ra.Context(chal)
    C, _ = ra.ra_sumcheck_matmul_prove(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
    want = A.astype(np.int64) @ B.astype(np.int64)  # |C| < 2^53: exact in int64
    assert np.array_equal(C.cpu().numpy(), want)


@pytest.mark.parametrize("m", [32, 256])  # the split launch (m < 64) and the fused front
def test_product_int32_top_plane(ra, m):
    """int32 rows whose entries all lie in [0, 2^24) have a zero top limb
    plane; a 64-row tile skips plane 3 only when all its rows do.  Tiles:
    such rows only (with 0, 2^24 - 1 and a zero row), one entry 2^24, one
    entry -1, and the full int32 range."""
    n, k = 256, 128
    rng = np.random.default_rng(7 + m)
    hi = (1 << 24) - 1
    A = rng.integers(0, hi, size=(n, m), dtype=np.int64, endpoint=True)
    A[0, :] = 0
    A[1, :] = hi
    A[2, 0] = hi
    A[64 + 5, 3] = 1 << 24
    A[128 + 63, m - 1] = -1
    A[192:, :] = rng.integers(-2 ** 31, 2 ** 31 - 1, size=(64, m), dtype=np.int64, endpoint=True)
    A = A.astype(np.int32)
    B = rng.integers(-32768, 32767, size=(m, k), dtype=np.int64, endpoint=True).astype(np.int16)
    B[:, 0] = -32768
    B[:, 1] = 32767
    chal = inputs.xorshift64_stream(31 + m, 512)
    ctx = ra.Context(chal)
    C, _ = ra.ra_sumcheck_matmul_prove(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
    want = A.astype(np.int64) @ B.astype(np.int64)
    assert np.array_equal(C.cpu().numpy(), want)


def test_two_register_passes_verified(ra):
    """2^23 outputs: the rounds over x take two register passes, and the plane
    rounds are evaluated by the second one's extra workgroups.  The oracle
    cannot prove a table this large, so the library's host verifier checks
    the transcript against the opened tables (every chain, final value and
    opening) and rejects a changed round word.  Synchronous and deferred runs
    (t given, witness announced) give the same transcript."""
    n, m, k = 2048, 64, 4096
    rng = np.random.default_rng(23)
    A = rng.integers(-2 ** 10, 2 ** 10, size=(n, m)).astype(np.int16)
    B = rng.integers(-2 ** 10, 2 ** 10, size=(m, k)).astype(np.int16)
    chal = inputs.xorshift64_stream(2323, 512)
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    g = ra.prove_layer(ra.Context(chal), Ad, Bd, 8, True, 0)
    tr = g["transcript"]
    assert tr["P"] == 64
    dctx = ra.Context(chal, deferred=True)
    gd = ra.prove_layer(dctx, Ad, Bd, 8, True, 0, tr["t"])
    dctx.sync()
    assert gd["transcript"] == tr
    L = dict(A=A, B=B, Z=g["Z"].cpu().numpy(), R=g["R"].cpu().numpy(), Rm=g["Rm"].cpu().numpy(),
             Y=g["Y"].cpu().numpy(), bits=g["bits"].cpu().numpy(), transcript=tr, chained=False)
    assert ra.ra_verify(chal, [L]) == (0, 0)
    ev = list(tr["rs_evals"])
    ev[0] = (int(ev[0]) + 1) % P61
    assert ra.ra_verify(chal, [dict(L, transcript=dict(tr, rs_evals=ev))])[0] != 0


@pytest.mark.parametrize("kind", ["int16", "int32_relu", "int32_full"])
def test_product_large_layer(ra, kind):
    """A 512 x 128 x 4096 layer (512 product tiles, two per CU, 2^21 outputs):
    C against numpy's exact int64 product.  int16 (ReLU) and int32_relu
    (every entry in [0, 2^24), so the tiles skip the top limb plane; no ReLU
    so that t stays within this path's limits) also run the witness fused
    into the epilogue (t given, deferred), checked against a numpy rescale,
    and the whole layer must be accepted by the host verifier (which opens A,
    B, R, Rm, Y, Z and checks the rounding link against the matrix claim).
    int32_full: entries over the whole int32 range with its extremes (t would
    exceed this path's limit of 29, so only the product is checked)."""
    n, m, k, s = 512, 128, 4096, 16
    rng = np.random.default_rng({"int16": 1, "int32_relu": 2, "int32_full": 3}[kind])
    if kind == "int16":
        A = rng.integers(-32768, 32768, size=(n, m)).astype(np.int16)
        A.flat[:2] = [-32768, 32767]
    elif kind == "int32_relu":
        A = rng.integers(0, 1 << 24, size=(n, m)).astype(np.int32)
    else:
        A = rng.integers(-(2 ** 31), 2 ** 31, size=(n, m), dtype=np.int64).astype(np.int32)
        A.flat[:3] = [-(2 ** 31), 2 ** 31 - 1, 0]
    B = rng.integers(-32768, 32768, size=(m, k)).astype(np.int16)
    B.flat[:2] = [-32768, 32767]
    Cw = A.astype(np.int64) @ B.astype(np.int64)            # |C| <= 128 * 2^46 fits int64
    seed = 0xC0FFEE + len(kind)
    if kind == "int32_full":
        ctx = ra.Context(seed=seed)
        C, _ = ra.ra_sumcheck_matmul_prove(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
        assert np.array_equal(C.cpu().numpy(), Cw)
        return
    relu = kind == "int16"
    half = 1 << (s - 1)
    R = (Cw + half) >> s                                     # nearest: floor((C + 2^(s-1)) / 2^s)
    u = np.where(R >= 0, R, -R - 1).max()
    t = max(0, int(u).bit_length() - 1)
    assert s + (t + 2) * (1 + relu) <= 64 and t <= 29
    ctx = ra.Context(seed=seed, deferred=True)
    g = ra.prove_layer(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), s, relu, 0, t)
    ctx.sync()
    assert np.array_equal(g["C"].cpu().numpy(), Cw)
    assert np.array_equal(g["R"].cpu().numpy().astype(np.int64), R)
    assert np.array_equal(g["Rm"].cpu().numpy().view(np.uint16).astype(np.int64), (Cw + half) & ((1 << s) - 1))
    assert np.array_equal(g["Z"].cpu().numpy().astype(np.int64), np.maximum(R, 0) if relu else R)
    L = dict(A=A, B=B, Z=g["Z"].cpu().numpy(), R=g["R"].cpu().numpy(), Rm=g["Rm"].cpu().numpy(),
             Y=g["Y"].cpu().numpy(), bits=g["bits"].cpu().numpy(), transcript=g["transcript"], chained=False)
    assert ra.ra_verify(seed, [L]) == (0, 0)


def test_product_wide_rows_fused_witness(ra):
    """A 2 x 16 x 2^23 layer: 64 rows of 8-byte outputs span 2^32 bytes, so the
    product's epilogue stores through full 64-bit addresses instead of 32-bit
    offsets from the tile's first entry.  The fused witness must equal numpy's
    rescale and the separate witness pass (plan=False), with identical
    transcripts."""
    n, m, k, s = 2, 16, 1 << 23, 12
    rng = np.random.default_rng(23)
    A = rng.integers(-32768, 32768, size=(n, m)).astype(np.int16)
    B = rng.integers(-32768, 32768, size=(m, k)).astype(np.int16)
    B[:, -1] = 32767
    A[0] = 32767
    Cw = A.astype(np.int64) @ B.astype(np.int64)             # |C| <= 16 * 2^30
    half = 1 << (s - 1)
    R = (Cw + half) >> s
    u = np.where(R >= 0, R, -R - 1).max()
    t = max(0, int(u).bit_length() - 1)
    assert s + 2 * (t + 2) <= 64 and t <= 29
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    seed = 0x5EED23
    ctx = ra.Context(seed=seed, deferred=True)
    g = ra.prove_layer(ctx, Ad, Bd, s, True, 0, t)
    ctx.sync()
    assert np.array_equal(g["C"].cpu().numpy(), Cw)
    Rg = g["R"].cpu().numpy().astype(np.int64)
    assert np.array_equal(Rg, R)
    assert np.array_equal(g["Rm"].cpu().numpy().view(np.uint16).astype(np.int64), (Cw + half) & ((1 << s) - 1))
    assert np.array_equal(g["Y"].cpu().numpy().astype(np.int64), np.abs(R))
    assert np.array_equal(g["Z"].cpu().numpy().astype(np.int64), np.maximum(R, 0))
    ctx2 = ra.Context(seed=seed, deferred=True)
    g2 = ra.prove_layer(ctx2, Ad, Bd, s, True, 0, t, plan=False)
    ctx2.sync()
    for key in ("R", "Rm", "Y", "Z", "bits"):
        assert torch.equal(g[key], g2[key]), key
    assert g["transcript"] == g2["transcript"]
