"""Deferred outputs (ra_ctx_set_deferred / ra_ctx_sync): the proving calls
return once enqueued and their host outputs are written at the sync.  The
transcripts and tables must equal the oracle's exactly, as in synchronous
mode; device-side errors surface at the sync."""
import numpy as np
import pytest
import torch

from helpers import diff_transcripts
from oracle import oracle as orc
from paper_2505_17623_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ra():
    from paper_2505_17623_amd import ra as ra_mod
    ra_mod.lib()
    assert torch.cuda.is_available()
    return ra_mod


def check_network(ra, got, want, label):
    for li, (g, o) in enumerate(zip(got, want)):
        bad = diff_transcripts(g["transcript"], o)
        assert not bad, f"{label} L{li}: transcript mismatch in {bad}"
        assert np.array_equal(g["C"].cpu().numpy(), o["C"]), f"{label} L{li} C"
        for key in ("R", "Y", "Z"):
            assert np.array_equal(g[key].cpu().numpy().astype(np.int64), o[key]), (label, li, key)
        planes = ra.unpack_bits(g["bits"].cpu().numpy(), g["transcript"]["P"])
        assert np.array_equal(planes, o["bits"]), f"{label} L{li} bits"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_deferred_with_given_t_matches_oracle(ra, cfg):
    wl = inputs.small(cfg)
    want = orc.prove_network(wl)
    ctx = ra.Context(wl.challenges, deferred=True)
    got = ra.prove_network(ctx, wl, ts=[o["t"] for o in want])
    assert got[0]["transcript"] == {}  # nothing is filled before the sync
    ctx.sync()
    check_network(ra, got, want, f"cfg{cfg}")
    assert ctx.cursor() == want[-1]["cursor"]


def test_deferred_without_t_waits_for_it(ra):
    wl = inputs.small(2)
    want = orc.prove_network(wl)
    ctx = ra.Context(wl.challenges, deferred=True)
    got = ra.prove_network(ctx, wl)
    ctx.sync()
    check_network(ra, got, want, "cfg2 t from data")


def test_two_networks_one_sync(ra):
    """Several layers' outputs pending at once (the staging area grows)."""
    wl = inputs.small(5)
    ref_ctx = ra.Context(wl.challenges)
    ref = ra.prove_network(ref_ctx, wl) + ra.prove_network(ref_ctx, wl)
    ts = [r["transcript"]["t"] for r in ref]
    ctx = ra.Context(wl.challenges, deferred=True)
    got = ra.prove_network(ctx, wl, ts=ts[:2]) + ra.prove_network(ctx, wl, ts=ts[2:])
    ctx.sync()
    for li, (g, r) in enumerate(zip(got, ref)):
        assert g["transcript"] == r["transcript"], f"layer {li}"
    assert ctx.cursor() == ref_ctx.cursor()


def test_deferred_range_error_at_sync(ra):
    chal = inputs.xorshift64_stream(77, 256)
    A = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    B = torch.full((4, 4), 3000, dtype=torch.int16).cuda()
    ctx = ra.Context(chal, deferred=True)
    C, _ = ra.ra_sumcheck_matmul_prove(ctx, A, B)
    (R, Rm, Y, Z, bits), info = ra.ra_rescale_relu_witness(ctx, C, 4, True, 0, t=3)  # R does not fit t = 3
    assert info.P == 16                                        # known on the host: 4 + 2 * (3 + 2) -> 16
    ra.ra_range_prove(ctx, bits, R, Y, info)
    with pytest.raises(ra.RAError) as e:
        ctx.sync()
    assert e.value.code == -4
    ctx.sync()  # the error is reported once


def test_planned_range_error_at_sync(ra):
    """The witness announced with a t that does not hold R: the error comes
    from the product's range flags, at the sync."""
    chal = inputs.xorshift64_stream(78, 256)
    A = torch.full((64, 64), 3000, dtype=torch.int16).cuda()
    B = torch.full((64, 64), 3000, dtype=torch.int16).cuda()
    ctx = ra.Context(chal, deferred=True)
    outs = ra.witness_outputs(64, 64, A.device)
    ra.ra_witness_plan(ctx, 4, True, 0, 3, outs)
    C, _ = ra.ra_sumcheck_matmul_prove(ctx, A, B)
    (R, Rm, Y, Z, bits), info = ra.ra_rescale_relu_witness(ctx, C, 4, True, 0, t=3, outs=outs)
    ra.ra_range_prove(ctx, bits, R, Y, info)
    with pytest.raises(ra.RAError) as e:
        ctx.sync()
    assert e.value.code == -4


@pytest.mark.parametrize("deferred", [False, True])
@pytest.mark.parametrize("change", ["outputs", "t", "relu"])
def test_plan_not_matching_runs_full_witness(ra, deferred, change):
    """A witness call whose arguments differ from the plan computes the
    witness itself; the transcript and tables equal the oracle's."""
    rng = np.random.default_rng(5)
    A = rng.integers(-2 ** 10, 2 ** 10, size=(128, 64)).astype(np.int16)
    B = rng.integers(-2 ** 10, 2 ** 10, size=(64, 128)).astype(np.int16)
    chal = inputs.xorshift64_stream(4321, 512)
    base = orc.prove_layer(A, B, 8, True, 0, chal)
    t_use = base["t"] + (1 if change == "t" else 0)
    relu = change != "relu"
    want = orc.prove_layer(A, B, 8, relu, 0, chal, t_in=t_use)
    ctx = ra.Context(chal, deferred=deferred)
    planned = ra.witness_outputs(128, 128, torch.device("cuda"))
    used = ra.witness_outputs(128, 128, torch.device("cuda")) if change == "outputs" else planned
    ra.ra_witness_plan(ctx, 8, True, 0, base["t"], planned)
    C, mm = ra.ra_sumcheck_matmul_prove(ctx, torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())
    (R, Rm, Y, Z, bits), info = ra.ra_rescale_relu_witness(ctx, C, 8, relu, 0, t_use, used)
    rs = ra.ra_range_prove(ctx, bits, R, Y, info)
    ctx.sync()
    tr = dict(mm)
    tr.update(rs)
    tr.update(t=int(info.t), P=int(info.P), r_claim=int(info.r_claim), rm_claim=int(info.rm_claim),
              y_claim=int(info.y_claim), z_claim=int(info.z_claim))
    bad = diff_transcripts(tr, want)
    assert not bad, f"{change}: transcript mismatch in {bad}"
    assert np.array_equal(Z.cpu().numpy().astype(np.int64), want["Z"])
    assert np.array_equal(ra.unpack_bits(bits.cpu().numpy(), tr["P"]), want["bits"])


def test_plan_state_and_arguments(ra):
    chal = inputs.xorshift64_stream(79, 256)
    A = torch.ones((4, 4), dtype=torch.int16).cuda()
    ctx = ra.Context(chal)
    outs = ra.witness_outputs(4, 4, A.device)
    with pytest.raises(ra.RAError) as e:
        ra.ra_witness_plan(ctx, 4, True, 0, -1, outs)      # t must be given
    assert e.value.code == -1
    with pytest.raises(ra.RAError) as e:
        ra.ra_witness_plan(ctx, 20, True, 0, 3, outs)      # s beyond this GPU path's 16
    assert e.value.code == -9
    ra.ra_sumcheck_matmul_prove(ctx, A, A)
    with pytest.raises(ra.RAError) as e:
        ra.ra_witness_plan(ctx, 4, True, 0, 3, outs)       # between a layer's calls
    assert e.value.code == -7
