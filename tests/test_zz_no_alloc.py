"""nitro_block_forward_noalloc (the entry point for callers that cannot allocate) against
nitro_block_forward, which the oracle-parity tests pin: the same block output, bit for bit, on
two calls in a row (the second with a smaller input, so that stale scratch contents from the
first call would show). The size limit is checked on the host (tests/test_abi.py)."""
import numpy as np
import pytest
import torch

from paper_2407_11698_amd import nitro as N

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)


def rand(rng, shape, lo, hi, dtype):
    return torch.from_numpy(rng.integers(lo, hi, size=shape, endpoint=True).astype(dtype)).to(DEV)


# (n, h, w, channels, pool, wmax): a pooled two-conv block on the tiled kernels (input padded to
# 16 channels), then the same block at a smaller batch; an unpooled block with multi-limb
# weights, then a smaller one; an MLP block
CASES = [
    [(8, 32, 32, [3, 64, 64], True, 44), (2, 32, 32, [3, 64, 64], True, 44)],
    [(4, 16, 16, [64, 128, 128], False, 6000), (1, 8, 8, [64, 128, 128], False, 6000)],
    [(64, 1, 1, [784, 100, 50], False, 300), (5, 1, 1, [784, 100, 50], False, 300)],
    # an MLP block whose full block state (about 80 MB) exceeds the 64 MiB array while its forward
    # part (about 52 MB, mostly the MFMA linear forward's split-K partials) fits
    [(4096, 1, 1, [64, 512, 512, 512, 512], False, 40), (1000, 1, 1, [64, 512, 512, 512, 512], False, 40)],
]


@pytest.mark.parametrize("calls", CASES, ids=["vgg_block", "wide_weights", "mlp", "mlp_big_state"])
def test_noalloc_matches_block_forward(calls):
    ctx = N.Context(0)
    try:
        rng = np.random.default_rng(7)
        for n, h, w, chans, pool, wmax in calls:
            print("noalloc case", dict(n=n, h=h, w=w, chans=chans, pool=pool), flush=True)
            conv = h > 1
            J = len(chans) - 1
            kind = N.CONV3X3 if conv else N.LINEAR
            desc = N.block_desc(n, h, w, [N.layer(kind, chans[j], chans[j + 1]) for j in range(J)],
                                pool, 0, 10)
            x = rand(rng, (n, h, w, chans[0]) if conv else (n, chans[0]), -127, 127, np.int8)
            ws = [rand(rng, (chans[j + 1], 3, 3, chans[j]) if conv else (chans[j + 1], chans[j]),
                       -wmax, wmax, np.int32) for j in range(J)]
            oh, ow = (h // 2, w // 2) if pool else (h, w)
            shape = (n, oh, ow, chans[-1]) if conv else (n, chans[-1])
            ref = torch.empty(shape, dtype=torch.int8, device=DEV)
            got = torch.full(shape, 77, dtype=torch.int8, device=DEV)
            state = torch.empty(N.block_query(desc), dtype=torch.uint8, device=DEV)
            if n == 4096:
                assert state.numel() > 64 << 20
            ctx.block_forward(desc, ws, x, ref, state)
            ctx.block_forward_noalloc(desc, ws, x, got)
            ctx.sync()
            assert torch.equal(ref, got)
    finally:
        ctx.close()
