"""nitro_preprocess (Appendix A integer normalisation) against the oracle: integer mean, mean
absolute deviation and every normalised byte, bit-exact, in both rounding modes; datasets of a
few bytes up to the CIFAR-10-sized synthetic set (153.6 M bytes); any alignment, in place; a
constant dataset (omega rounds to 0) and values that saturate int8."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2407_11698_amd import nitro as N
from paper_2407_11698_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)
MODES = [(N.ROUND_FLOOR, O.FLOOR), (N.ROUND_TRUNC, O.TRUNC)]


@pytest.fixture(scope="module")
def ctx():
    c = N.Context(0)
    yield c
    c.close()


def run(ctx, x: np.ndarray, nm, offset=0, inplace=False):
    """The library on x (placed `offset` bytes into a buffer), compared with the oracle."""
    print("preprocess case", dict(count=x.size, offset=offset, inplace=inplace, mode=nm), flush=True)
    buf = torch.zeros(x.size + offset + 16, dtype=torch.uint8, device=DEV)
    xd = buf[offset:offset + x.size]
    xd.copy_(torch.from_numpy(x.reshape(-1)))
    out = xd.view(torch.int8) if inplace else torch.full((x.size,), 99, dtype=torch.int8, device=DEV)
    stats = torch.zeros(3, dtype=torch.int64, device=DEV)
    ws = torch.empty(N.preprocess_query(x.size), dtype=torch.uint8, device=DEV)
    ws.fill_(0xAB)
    ctx.preprocess(xd, out, stats, ws, nm)
    ctx.sync()
    return out.cpu().numpy(), stats.cpu().numpy()


@pytest.mark.parametrize("count,offset", [(1, 0), (15, 3), (16, 0), (17, 1), (1000, 7),
                                          (16 * 4096 * 4 + 5, 0), (16 * 4096 * 4 + 5, 9),
                                          (3 * 1024 * 2000, 0)])
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_preprocess_sizes(ctx, count, offset, modes):
    x = WL.draw_image_bytes((count,), seed=count + offset)
    got, st = run(ctx, x, modes[0], offset)
    ref = O.preprocess(x, modes[1])
    assert st.tolist() == [ref.mu, ref.omega, ref.saturated]
    assert np.array_equal(got, ref.xhat)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_preprocess_in_place_and_edges(ctx, modes):
    x = WL.draw_image_bytes((5000, 3), seed=3)
    got, st = run(ctx, x, modes[0], offset=5, inplace=True)
    ref = O.preprocess(x, modes[1])
    assert np.array_equal(got, ref.xhat) and st.tolist() == [ref.mu, ref.omega, ref.saturated]
    # constant data (omega rounds to 0, divided by 1) and a dataset whose extremes saturate
    for x in (np.full(777, 42, np.uint8), np.array([7, 7, 7, 8] * 50, np.uint8),
              np.concatenate([np.zeros(1000, np.uint8), np.full(3, 255, np.uint8)])):
        got, st = run(ctx, x, modes[0])
        ref = O.preprocess(x, modes[1])
        assert np.array_equal(got, ref.xhat) and st.tolist() == [ref.mu, ref.omega, ref.saturated]


def test_preprocess_cifar_sized(ctx):
    """The full synthetic CIFAR-10-sized dataset (50000 x 32 x 32 x 3 bytes), as the benchmark
    normalises it."""
    x = WL.draw_image_bytes(WL.CIFAR10_BYTES, seed=0)
    got, st = run(ctx, x, N.ROUND_FLOOR)
    ref = O.preprocess(x, O.FLOOR)
    assert st.tolist() == [ref.mu, ref.omega, ref.saturated]
    assert np.array_equal(got, ref.xhat)


def test_preprocess_rejects_bad_arguments(ctx):
    x = torch.zeros(16, dtype=torch.uint8, device=DEV)
    out = torch.zeros(16, dtype=torch.int8, device=DEV)
    st = torch.zeros(3, dtype=torch.int64, device=DEV)
    ws = torch.zeros(N.preprocess_query(16), dtype=torch.uint8, device=DEV)
    assert N.LIB.nitro_preprocess(ctx.h, x.data_ptr(), 0, 0, out.data_ptr(), st.data_ptr(), ws.data_ptr()) == N.EINVAL
    assert N.LIB.nitro_preprocess(ctx.h, x.data_ptr(), 16, 7, out.data_ptr(), st.data_ptr(), ws.data_ptr()) == N.EINVAL
    assert N.LIB.nitro_preprocess(ctx.h, x.data_ptr(), 16, 0, out.data_ptr(), None, ws.data_ptr()) == N.EINVAL
    ctx.sync()
