"""ra_mle_bind_noalloc (fixed device scratch, no allocation) against
ra_mle_bind through the C ABI: bit-identical outputs, on two calls in a row
with the second smaller, on the current stream and on a second stream."""
import numpy as np
import pytest
import torch

from paper_2505_17623_amd import inputs

pytestmark = pytest.mark.gpu
P61 = (1 << 61) - 1


@pytest.fixture(scope="module")
def ra():
    from paper_2505_17623_amd import ra as ra_mod
    ra_mod.lib()
    assert torch.cuda.is_available()
    return ra_mod


def table(shape, dt, seed):
    rng = np.random.default_rng(seed)
    if dt == "field":
        T = rng.integers(0, P61, size=shape, dtype=np.uint64)
        return torch.from_numpy(T.view(np.int64)).cuda()
    if dt == np.int64:
        return torch.from_numpy(rng.integers(-(2 ** 62), 2 ** 62, size=shape, dtype=np.int64)).cuda()
    info = np.iinfo(dt)
    return torch.from_numpy(rng.integers(info.min, info.max, size=shape, dtype=dt, endpoint=True)).cuda()


@pytest.mark.parametrize("dt", [np.int16, np.int32, np.int64, "field"])
@pytest.mark.parametrize("bind_rows", [True, False])
def test_noalloc_matches_mle_bind(ra, dt, bind_rows):
    ctx = ra.Context(inputs.xorshift64_stream(5, 8))
    side = torch.cuda.Stream()
    for i, shape in enumerate([(1024, 512), (64, 32), (8, 2048), (1, 1)]):
        T = table(shape, dt, 100 * i + 7)
        rows, cols = shape
        v = (rows if bind_rows else cols).bit_length() - 1
        z = [int(x) for x in inputs.xorshift64_stream(90 + v + i, max(v, 1))[:v]]
        want = ra.ra_mle_bind(ctx, T, bind_rows, z, field=(dt == "field")).cpu()
        for stream in (None, side):
            out = torch.full((cols if bind_rows else rows,), -1, dtype=torch.int64, device="cuda")
            if stream is not None:
                stream.wait_stream(torch.cuda.current_stream())
            ra.ra_mle_bind_noalloc(T, bind_rows, z, out, field=(dt == "field"), stream=stream)
            (stream or torch.cuda.current_stream()).synchronize()
            assert torch.equal(out.cpu(), want), (dt, bind_rows, shape, stream is not None)
    ctx.close()


def test_noalloc_largest_table(ra):
    """The largest row binding the scratch holds (2^18 rows: a 2 MiB eq
    table plus the chunk sums), then a small one."""
    ctx = ra.Context(inputs.xorshift64_stream(5, 8))
    for shape in [(1 << 18, 4), (16, 4)]:
        T = table(shape, np.int16, shape[0])
        v = shape[0].bit_length() - 1
        z = [int(x) for x in inputs.xorshift64_stream(77 + v, v)]
        want = ra.ra_mle_bind(ctx, T, True, z).cpu()
        out = torch.empty(shape[1], dtype=torch.int64, device="cuda")
        ra.ra_mle_bind_noalloc(T, True, z, out)
        torch.cuda.synchronize()
        assert torch.equal(out.cpu(), want), shape
    ctx.close()
