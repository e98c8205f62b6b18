"""The int8 matrix-core rate probe (nitro_mfma_rate) through the C ABI: argument checks, and a
rate that is positive and not above the published dense int8 peak of the MI355X (5.0 * 10^15
ops/s; a higher figure would mean the probe's op count is wrong)."""
import pytest

from paper_2407_11698_amd import nitro as N

pytestmark = pytest.mark.gpu

PUBLISHED_INT8_TOPS = 5000.0


@pytest.fixture(scope="module")
def ctx():
    c = N.Context(0)
    yield c
    c.close()


@pytest.mark.parametrize("waves,iters", [(0, 100), (5, 100), (2, 0)])
def test_mfma_rate_rejects_bad_counts(ctx, waves, iters):
    with pytest.raises(N.NitroError) as e:
        ctx.mfma_rate(waves, iters)
    assert e.value.code == N.EINVAL


@pytest.mark.parametrize("waves", [1, 2])
def test_mfma_rate_within_published_peak(ctx, waves):
    tops = ctx.mfma_rate(waves, 4000)
    print("int8 MFMA rate, %d waves per SIMD: %.0f TOP/s" % (waves, tops), flush=True)
    assert 0.0 < tops <= PUBLISHED_INT8_TOPS * 1.02
