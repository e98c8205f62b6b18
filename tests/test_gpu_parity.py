"""GPU parity: the HIP library (through the C ABI) against the CPU oracle, element by element and
bit-exact, on seeded inputs. Block-level calls at shapes that span several tiles and ragged
tails, the edge cases of the method, IntegerSGD, the output layer and whole training steps."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2407_11698_amd import nitro as N
from paper_2407_11698_amd import runner
from paper_2407_11698_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)
MODES = [(N.ROUND_FLOOR, O.FLOOR), (N.ROUND_TRUNC, O.TRUNC)]


@pytest.fixture(scope="module")
def ctx():
    c = N.Context(0)
    yield c
    c.close()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def rand(rng, shape, lo, hi, dtype):
    return rng.integers(lo, hi, size=shape, endpoint=True).astype(dtype)


def run_block(ctx, rng, n, h, w, chans, maxpool, G, alpha, nm, om, wmax=127, dmax=1 << 15,
              conv=True, tap_last_g=True, d_lr=0, tap_inner_g=True, delta_edit=None):
    """One nitro_block_forward + nitro_block_backward against the oracle's block functions.
    tap_last_g=False leaves the last layer's g untapped (the library may then keep it pooled);
    tap_inner_g=False the other layers' (the library may then keep them in 16 bits with escapes).
    delta_edit(rng, delta, rec) (no learning layer): the given delta, edited after the forward.
    Returns the oracle's record."""
    print("block case", dict(n=n, h=h, w=w, chans=chans, pool=maxpool, G=G, alpha=alpha,
                             mode=nm, wmax=wmax, conv=conv), flush=True)
    J = len(chans) - 1
    if conv:
        x = rand(rng, (n, h, w, chans[0]), -127, 127, np.int8)
        ws = [rand(rng, (chans[j + 1], 3, 3, chans[j]), -wmax, wmax, np.int32) for j in range(J)]
        layers = [N.layer(N.CONV3X3, chans[j], chans[j + 1]) for j in range(J)]
        hh, ww = h, w
    else:
        x = rand(rng, (n, chans[0]), -127, 127, np.int8)
        ws = [rand(rng, (chans[j + 1], chans[j]), -wmax, wmax, np.int32) for j in range(J)]
        layers = [N.layer(N.LINEAR, chans[j], chans[j + 1]) for j in range(J)]
        hh = ww = 1
    desc = N.block_desc(n, hh, ww, layers, maxpool, G, alpha, nm, d_lr)
    # oracle
    rec = O.block_forward(x, ws, maxpool, alpha, om)
    out_shape = rec.out.shape
    f = rec.out
    win = (1, 1)
    if conv and G and d_lr:
        win = O.learning_pool_window(out_shape[3], out_shape[1], out_shape[2], d_lr)
        if win != (1, 1):
            f, f_idx = O.maxpool_window(rec.out, *win)
    f_shape = f.shape
    d = int(np.prod(f_shape[1:]))
    labels = rng.integers(0, max(G, 1), n).astype(np.int32)
    want_dx, expect_overflow = True, False
    w_lr = rand(rng, (G, d), -wmax, wmax, np.int32) if G else None
    delta = None if G else rand(rng, out_shape, -dmax, dmax, np.int32)
    if delta_edit is not None:
        delta = delta_edit(rng, delta, rec)
    try:
        if G > 0:
            ff = f.reshape(n, d)
            rec.yhat = O.learning_forward(ff, w_lr, om)
            rec.e = O.check_int32(O.loss_grad(rec.yhat, labels, G), "e")
            rec.dw_lr = O.linear_dw(rec.e, ff)
            rec.delta_fw = O.check_int32(O.linear_dx(rec.e, w_lr), "delta")
            delta = rec.delta_fw.reshape(f_shape)
            if win != (1, 1):
                delta = O.maxpool_window_bwd(delta, f_idx, out_shape, *win)
        try:
            O.block_backward(rec, ws, delta, maxpool, alpha, om, want_dx=True)
        except OverflowError:
            want_dx = False              # only the optional input gradient may be out of range
            O.block_backward(rec, ws, delta, maxpool, alpha, om, want_dx=False)
    except OverflowError:
        expect_overflow = True
    # GPU
    xd = dev(x)
    wd = [dev(a) for a in ws]
    a_out = torch.empty(out_shape, dtype=torch.int8, device=DEV)
    state = torch.empty(N.block_query(desc), dtype=torch.uint8, device=DEV)
    ctx.block_forward(desc, wd, xd, a_out, state)
    dws = [torch.empty(a.shape, dtype=torch.int64, device=DEV) for a in ws]
    dw_lr = torch.empty((G, d), dtype=torch.int64, device=DEV) if G else None
    taps = {"g": [torch.empty(l.zs.shape, dtype=torch.int32, device=DEV)
                  if (tap_last_g if j == J - 1 else tap_inner_g) else None
                  for j, l in enumerate(rec.layers)],
            "dx": torch.empty(x.shape, dtype=torch.int64, device=DEV) if want_dx else None}
    if G:
        taps["yhat"] = torch.empty((n, G), dtype=torch.int32, device=DEV)
        taps["e"] = torch.empty((n, G), dtype=torch.int32, device=DEV)
        taps["delta"] = torch.empty(f_shape, dtype=torch.int32, device=DEV)
    ctx.block_backward(desc, wd, dev(w_lr) if G else None, xd, a_out,
                       dev(labels) if G else None, None if G else dev(delta), state, dws, dw_lr,
                       taps)
    if expect_overflow:
        assert ctx.sync_status() == N.EOVERFLOW
        return rec
    ctx.sync()
    assert np.array_equal(host(a_out), rec.out), "block output"
    if G:
        assert np.array_equal(host(taps["yhat"]), rec.yhat), "yhat"
        assert np.array_equal(host(taps["e"]), rec.e), "e"
        assert np.array_equal(host(dw_lr), rec.dw_lr), "dW learning"
        assert np.array_equal(host(taps["delta"]), rec.delta_fw.reshape(f_shape)), "delta_fw"
    for j in range(J):
        if taps["g"][j] is not None:
            assert np.array_equal(host(taps["g"][j]), rec.g[j]), "g layer %d" % j
        assert np.array_equal(host(dws[j]), rec.dw[j]), "dW layer %d" % j
    if want_dx:
        assert np.array_equal(host(taps["dx"]), rec.dx), "dx"
    return rec


CONV_CASES = [
    # n, h, w, chans, pool, G, alpha, wmax
    (2, 6, 6, [1, 16], True, 10, 10, 127),
    (3, 10, 6, [3, 32], True, 10, 10, 127),
    (2, 4, 4, [5, 7, 9], True, 3, 10, 127),
    (2, 8, 8, [16, 32, 16], False, 0, 10, 127),
    (1, 2, 2, [4, 4], True, 2, 2, 2000),
    (2, 5, 7, [6, 5], False, 4, 3, 30000),
    (2, 6, 10, [64, 64], True, 10, 10, 127),
    (1, 4, 4, [128, 256], True, 100, 10, 9),
    (2, 8, 8, [64, 128, 128], True, 100, 16, 6000),
    (1, 32, 32, [3, 64, 64], True, 100, 10, 44),
    # one-pixel-high and 1x1 images: every tap but the centre (or the centre row) in the padding
    (3, 1, 5, [16, 16], False, 4, 10, 127),
    (2, 1, 1, [8, 32, 16], False, 10, 10, 127),
]


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block(ctx, case, modes):
    n, h, w, chans, pool, G, alpha, wmax = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G)) % (1 << 31))
    run_block(ctx, rng, n, h, w, chans, pool, G, alpha, modes[0], modes[1], wmax=wmax)


# shapes the tiled conv kernels take with either tile (128 or 256 output pixels per workgroup):
# whole small images per tile, image rows per tile, multi-limb weights, with and without pooling
TILE_CASES = [
    (2, 8, 8, [64, 128, 128], True, 100, 16, 6000),
    (1, 32, 32, [3, 64, 64], True, 100, 10, 44),
    (3, 16, 16, [32, 64, 64], True, 10, 10, 300),
    (2, 16, 16, [64, 64, 64], False, 0, 10, 127),
]


@pytest.mark.parametrize("tile", [128, 256])
@pytest.mark.parametrize("case", TILE_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_tile(ctx, tile, case, modes):
    """The same block results whichever conv tile is forced (nitro_set_conv_tile)."""
    n, h, w, chans, pool, G, alpha, wmax = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G, tile)) % (1 << 31))
    ctx.set_conv_tile(tile)
    try:
        run_block(ctx, rng, n, h, w, chans, pool, G, alpha, modes[0], modes[1], wmax=wmax)
    finally:
        ctx.set_conv_tile(0)


# persistent 256-pixel workgroups (about 4 tiles each): 1 workgroup on 2 to 4 tiles, 3 on 10
# (ragged), 2 on 8 (the XCD-ordered tile map), with and without pooling and weight limbs
PERSIST_CASES = [
    (3, 16, 16, [32, 64, 64], True, 10, 10, 300),
    (5, 16, 16, [64, 128, 128], True, 100, 16, 6000),
    (8, 16, 16, [32, 64, 64], False, 0, 10, 127),
    (1, 32, 32, [3, 64, 64], True, 100, 10, 44),
]


@pytest.mark.parametrize("case", PERSIST_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_persistent(ctx, case, modes):
    """The same block results with persistent conv workgroups (nitro_set_conv_persistent)."""
    n, h, w, chans, pool, G, alpha, wmax = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G, 9001)) % (1 << 31))
    ctx.set_conv_tile(256)
    ctx.set_conv_persistent(1)
    try:
        run_block(ctx, rng, n, h, w, chans, pool, G, alpha, modes[0], modes[1], wmax=wmax)
    finally:
        ctx.set_conv_tile(0)
        ctx.set_conv_persistent(0)


# pooled blocks on the MFMA learning layer whose last layer's g is not tapped: the learning layer
# leaves that g pooled and the weight-gradient planes un-pool it (one and two conv layers, both
# conv tiles)
POOLED_G_CASES = [
    (2, 8, 8, [64, 128, 128], True, 100, 16, 6000),
    (1, 32, 32, [3, 64, 64], True, 100, 10, 44),
    (3, 16, 16, [32, 64, 64], True, 10, 10, 300),
    (2, 6, 10, [64, 64], True, 10, 10, 127),
]


@pytest.mark.parametrize("tile", [128, 256])
@pytest.mark.parametrize("case", POOLED_G_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_pooled_g(ctx, tile, case, modes):
    n, h, w, chans, pool, G, alpha, wmax = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G, tile, 77)) % (1 << 31))
    ctx.set_conv_tile(tile)
    try:
        run_block(ctx, rng, n, h, w, chans, pool, G, alpha, modes[0], modes[1], wmax=wmax,
                  tap_last_g=False)
    finally:
        ctx.set_conv_tile(0)


# weight gradients of wide layers (256 to 512 output channels, 64-channel tiles x 16-channel input
# tiles): g in 1 to 4 limbs, one K split (dW written directly) and several (int64 partials), a
# partial output-channel tile with C_in % 16 != 0, pooled and not; the last two cases have at
# least 32 super-steps per workgroup, where g in 3 limbs takes all four waves of a workgroup
WIDE_DW_CASES = [
    # n, h, w, chans, pool, dmax
    (2, 6, 6, [256, 256], False, 100),
    (2, 6, 6, [256, 256], True, 5000),
    (2, 6, 6, [32, 256, 256], False, 1 << 15),
    (1, 4, 4, [256, 256], False, 1 << 24),
    (1, 4, 4, [250, 272], False, 1 << 15),
    (8, 16, 16, [256, 256], True, 5000),
    (16, 32, 32, [256, 512], False, 1 << 15),
    (16, 32, 32, [256, 512], False, 5000),
]


@pytest.mark.parametrize("case", WIDE_DW_CASES)
def test_conv_block_wide_weight_gradient(ctx, case):
    n, h, w, chans, pool, dmax = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), dmax, 4242)) % (1 << 31))
    run_block(ctx, rng, n, h, w, chans, pool, 0, 10, N.ROUND_FLOOR, O.FLOOR, dmax=dmax)


# blocks whose inner layers' gradients are not tapped, on the tiled input gradient and the planes
# weight gradient: g_{j-1} is then kept in 16 bits with escapes for |g| > 32767 (the last flag:
# whether the oracle's inner gradients have such values, checked); the four-layer case passes the
# 16-bit form down twice
G16_CASES = [
    # n, h, w, chans, pool, G, alpha, wmax, dmax, escapes
    (1, 32, 32, [3, 64, 64], True, 100, 10, 2, 0, False),
    (3, 16, 16, [32, 64, 64], True, 10, 10, 3, 0, False),
    (2, 8, 8, [64, 128, 128], True, 100, 16, 4, 0, False),
    (3, 16, 16, [32, 64, 64], True, 10, 10, 300, 0, True),
    (2, 16, 16, [64, 64, 64], False, 0, 10, 1, 300, False),
    (2, 16, 16, [64, 64, 64], False, 0, 10, 2, 1000, True),
    (2, 16, 16, [64, 64, 64], False, 0, 10, 3, 3000, True),
    (2, 16, 16, [64, 64, 64, 64], False, 0, 10, 1, 16, False),
    (2, 16, 16, [64, 64, 64, 64], False, 0, 10, 2, 1000, True),
]


@pytest.mark.parametrize("case", G16_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_inner_g16(ctx, case, modes):
    n, h, w, chans, pool, G, alpha, wmax, dmax, escapes = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G, wmax, 16)) % (1 << 31))
    rec = run_block(ctx, rng, n, h, w, chans, pool, G, alpha, modes[0], modes[1], wmax=wmax,
                    tap_inner_g=False, dmax=max(dmax, 1))
    inner = [np.abs(np.asarray(g, dtype=np.int64)).max() for g in rec.g[:-1]]
    assert (max(inner) > 32767) == escapes, inner


# The first layer's int64 input gradient with g one value past two limbs (32639 < max|g| <=
# 32768): the library takes g - 128 in two limbs, adds the offset's term per border class and
# corrects each g = 32768 from a list (more than 16384 of them: three limbs instead); so does the
# weight gradient where it is split (C_in a multiple of 64), with x's window sums as the term. The given
# delta is drawn in [-32767, 32767] and then set to 32768 at `plus` positions where NITRO-ReLU
# passes it unchanged (z* in [0, 127]) and to -32768 at 5 such positions; top = 32769 puts one
# 32769 there instead (outside the offset range), top = 32000 draws no edit at all.
G_OFFSET_CASES = [
    # n, h, w, chans, pool, plus, top
    (4, 16, 16, [64, 64], False, 0, 32768),
    (4, 16, 16, [64, 64], False, 7, 32768),
    (4, 16, 16, [64, 64], False, 300, 32768),
    (8, 16, 16, [64, 64], False, 16484, 32768),
    (3, 8, 8, [32, 32], False, 40, 32768),
    (2, 4, 4, [16, 16], False, 9, 32768),
    (2, 16, 2, [16, 16], False, 9, 32768),
    (2, 8, 8, [16, 32], True, 0, 32768),
    (4, 16, 16, [64, 64], False, 7, 32769),
    (4, 16, 16, [64, 64], False, 0, 32000),
    # split-K weight gradients with C_in % 64 == 0: the weight gradient takes the form too
    (16, 16, 16, [64, 64], False, 0, 32768),
    (16, 16, 16, [64, 64], False, 11, 32768),
    (8, 32, 32, [128, 64], False, 200, 32768),
    (16, 16, 16, [64, 64], False, 20000, 32768),
    (16, 8, 32, [64, 128], False, 60, 32768),
]


def g_offset_edit(plus, top):
    def edit(rng, delta, rec):
        if top == 32000:
            return np.clip(delta, -32000, 32000).astype(np.int32)
        d = np.clip(delta, -32767, 32767).astype(np.int32)
        zs = np.asarray(rec.layers[-1].zs)
        if zs.shape != d.shape:        # pooled: the random draw reaches the range by itself
            return rand(rng, d.shape, -32768, 32768, np.int32)
        idx = np.flatnonzero((zs >= 0) & (zs <= 127))
        pick = rng.choice(idx, size=plus + 5 + 1, replace=False)
        flat = d.reshape(-1)
        flat[pick[:plus]] = 32768 if top == 32768 else 0
        flat[pick[plus:plus + 5]] = -32768
        if top == 32769:
            flat[pick[-1]] = 32769
        return d
    return edit


@pytest.mark.parametrize("tap", [True, False], ids=["g_tapped", "g_untapped"])
@pytest.mark.parametrize("tile", [128, 256])
@pytest.mark.parametrize("case", G_OFFSET_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_g_offset(ctx, tile, case, modes, tap):
    """(g untapped and not pooled: the ReLU' pass hands g to the weight-gradient preparation in
    16 bits, its +-32768 escaped)"""
    n, h, w, chans, pool, plus, top = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), pool, plus, top, 128)) % (1 << 31))
    ctx.set_conv_tile(tile)
    try:
        rec = run_block(ctx, rng, n, h, w, chans, pool, 0, 10, modes[0], modes[1],
                        delta_edit=g_offset_edit(plus, top), tap_last_g=tap)
    finally:
        ctx.set_conv_tile(0)
    g = np.asarray(rec.g[0], dtype=np.int64)
    if not pool:
        assert int(np.abs(g).max()) == (top if top != 32000 else int(np.abs(g).max()))
        assert int((g == 32768).sum()) == (plus if top == 32768 else 0)


# nitro_layer_forward / nitro_layer_backward: one layer (a one-layer block with no pooling and
# no learning layer) against the oracle's block functions, with and without the g and dx
# outputs; the 64-channel conv case draws delta up to 32768 (g in the offset form when dx is
# asked for).
LAYER_CASES = [
    # kind, n, h, w, c_in, c_out, dmax
    (N.CONV3X3, 2, 8, 8, 16, 32, 1 << 15),
    (N.CONV3X3, 3, 7, 5, 3, 16, 5000),
    (N.CONV3X3, 16, 16, 16, 64, 64, 1 << 15),
    (N.LINEAR, 16, 1, 1, 100, 50, 1 << 15),
]


@pytest.mark.parametrize("outs", ["all", "none"])
@pytest.mark.parametrize("case", LAYER_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_layer_calls(ctx, case, modes, outs):
    kind, n, h, w, ci, co, dmax = case
    print("layer case", case, modes[0], outs, flush=True)
    rng = np.random.default_rng(hash((kind, n, h, w, ci, co, dmax, 77)) % (1 << 31))
    conv = kind == N.CONV3X3
    xs = (n, h, w, ci) if conv else (n, ci)
    ws = (co, 3, 3, ci) if conv else (co, ci)
    x = rand(rng, xs, -127, 127, np.int8)
    wt = rand(rng, ws, -127, 127, np.int32)
    rec = O.block_forward(x, [wt], False, 10, modes[1])
    delta = rand(rng, rec.out.shape, -dmax, dmax, np.int32)
    O.block_backward(rec, [wt], delta, False, 10, modes[1], want_dx=True)
    desc = N.layer_desc(n, h if conv else 1, w if conv else 1, N.layer(kind, ci, co), 10, modes[0])
    state = torch.empty(N.layer_query(desc), dtype=torch.uint8, device=DEV)
    xd, wd = dev(x), dev(wt)
    a_out = torch.empty(rec.out.shape, dtype=torch.int8, device=DEV)
    ctx.layer_forward(desc, wd, xd, a_out, state)
    dw = torch.empty(wt.shape, dtype=torch.int64, device=DEV)
    g = torch.empty(rec.out.shape, dtype=torch.int32, device=DEV) if outs == "all" else None
    dx = torch.empty(x.shape, dtype=torch.int64, device=DEV) if outs == "all" else None
    ctx.layer_backward(desc, wd, xd, a_out, dev(delta), state, dw, g, dx)
    ctx.sync()
    assert np.array_equal(host(a_out), rec.out), "output"
    assert np.array_equal(host(dw), rec.dw[0]), "dW"
    if outs == "all":
        assert np.array_equal(host(g), rec.g[0]), "g"
        assert np.array_equal(host(dx), rec.dx), "dx"


# (the forward layers and their weight gradients run on the int8 MFMA GEMM with K zero-padded
# to 16: 100, 50, 37, 3000 are ragged; 3000 and the split-K forward are MLP 4's widths; a batch
# of one with one output unit, and one input feature)
@pytest.mark.parametrize("chans,G,wmax,n", [([784, 100], 10, 7, 64), ([100, 50, 30], 10, 300, 5),
                                            ([37, 5], 3, 20000, 5), ([64, 65], 0, 127, 5),
                                            ([1024, 3000], 10, 40, 16), ([3000, 3000], 10, 3000, 7),
                                            ([3000, 1000, 200], 0, 127, 3), ([17, 1], 2, 127, 1),
                                            ([1, 16], 3, 127, 2)])
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_linear_block(ctx, chans, G, wmax, n, modes):
    rng = np.random.default_rng(len(chans) * 1000 + chans[0] + chans[1])
    run_block(ctx, rng, n, 1, 1, chans, False, G, 10, modes[0], modes[1], wmax=wmax, conv=False)


# conv blocks whose learning layer reads the block output max-pooled to at most d_lr features
# (windows (4, 2), (2, 2), (8, 4), (1, 2) with an odd height, none), pooled and unpooled blocks,
# one and two conv layers
LR_POOL_CASES = [
    # n, h, w, chans, pool, G, d_lr
    (2, 8, 8, [16, 32], True, 10, 64),
    (3, 8, 8, [16, 32], False, 10, 512),
    (2, 32, 32, [3, 128], False, 10, 4096),
    (1, 5, 6, [8, 16], False, 4, 250),
    (2, 16, 16, [32, 64, 64], True, 10, 1024),
    (2, 8, 8, [16, 32], True, 10, 100000),
    (2, 8, 8, [16, 6], False, 10, 64),       # 6 channels: the one-channel-per-thread kernels
]


@pytest.mark.parametrize("case", LR_POOL_CASES)
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_block_learning_pool(ctx, case, modes):
    n, h, w, chans, pool, G, d_lr = case
    rng = np.random.default_rng(hash((n, h, w, tuple(chans), G, d_lr)) % (1 << 31))
    run_block(ctx, rng, n, h, w, chans, pool, G, 10, modes[0], modes[1], wmax=300, d_lr=d_lr)


def test_gradient_overflow_is_flagged(ctx):
    """A block whose error signal cannot fit int32: the oracle raises, the GPU flags it."""
    rng = np.random.default_rng(77)
    run_block(ctx, rng, 2, 6, 6, [32, 32, 32], False, 0, 10, N.ROUND_FLOOR, O.FLOOR,
              wmax=1 << 20, dmax=1 << 15)


@pytest.mark.parametrize("alpha", [2, 3, 4, 5, 8, 64, 100, 127, 128])
def test_relu_alphas(ctx, alpha):
    """Every NITRO-ReLU segment, for many alpha_inv: int16-range weights saturate both ends."""
    rng = np.random.default_rng(alpha)
    run_block(ctx, rng, 2, 6, 6, [8, 12], False, 0, alpha, N.ROUND_FLOOR, O.FLOOR, wmax=20000)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_sgd(ctx, modes):
    rng = np.random.default_rng(5)
    w = rand(rng, (100003,), -(1 << 24), 1 << 24, np.int32)
    for gamma, lam, eta in [(512, 3000, -1), (327680, 25000, -1), (1, 0, -1), (4, 3, -1),
                            (3276800, 25000, 1000)]:
        dw = rand(rng, (100003,), -gamma << 20, gamma << 20, np.int64)
        ref = O.integer_sgd(w, dw, gamma, lam, modes[1], eta)
        wd = dev(w)
        ctx.integer_sgd_step(wd, dev(dw), gamma, lam, eta, modes[0])
        ctx.sync()
        assert np.array_equal(host(wd), ref), (gamma, lam, eta)


def test_sgd_overflow_flag(ctx):
    w = np.array([(1 << 31) - 1, 5], np.int32)
    dw = np.array([-1, 0], np.int64)
    wd = dev(w)
    ctx.integer_sgd_step(wd, dev(dw), 1, 0)
    assert ctx.sync_status() == N.EOVERFLOW
    assert host(wd)[0] == (1 << 31) - 1
    assert ctx.sync_status() == N.OK                   # the flag is cleared by reading it


def test_label_flag(ctx):
    n, d, G = 4, 8, 3
    f = dev(np.ones((n, d), np.int8))
    w = dev(np.ones((G, d), np.int32))
    labels = dev(np.array([0, 1, 3, 2], np.int32))
    dw = torch.empty((G, d), dtype=torch.int64, device=DEV)
    yhat = torch.empty((n, G), dtype=torch.int32, device=DEV)
    e = torch.empty((n, G), dtype=torch.int32, device=DEV)
    ctx.head_backward(n, d, G, f, w, labels, N.ROUND_FLOOR, dw, yhat, e)
    assert ctx.sync_status() == N.ELABEL


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_head(ctx, modes):
    rng = np.random.default_rng(9)
    n, d, G = 64, 2048, 10
    f = rand(rng, (n, d), -87, 104, np.int8)
    w = rand(rng, (G, d), -3000, 3000, np.int32)
    labels = rng.integers(0, G, n).astype(np.int32)
    yhat = O.learning_forward(f, w, modes[1])
    e = O.loss_grad(yhat, labels, G)
    dw_ref = O.linear_dw(e, f)
    dw = torch.empty((G, d), dtype=torch.int64, device=DEV)
    yd = torch.empty((n, G), dtype=torch.int32, device=DEV)
    ed = torch.empty((n, G), dtype=torch.int32, device=DEV)
    ctx.head_backward(n, d, G, dev(f), dev(w), dev(labels), modes[0], dw, yd, ed)
    ctx.sync()
    assert np.array_equal(host(yd), yhat)
    assert np.array_equal(host(ed), e)
    assert np.array_equal(host(dw), dw_ref)


# ------------------------------------------------------------------ whole training iterations

def oracle_net(wl, weights, om):
    hp = O.Hyper(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr, wl.alpha_inv, wl.n_classes,
                 mode=om, af_classes=wl.af_classes, d_lr=wl.d_lr,
                 dropout_conv_ppm=wl.dropout_conv_ppm, dropout_lin_ppm=wl.dropout_lin_ppm,
                 dropout_seed=wl.dropout_seed)
    specs = [(len(b.layers), b.maxpool, b.learning) for b in wl.blocks]
    return O.OracleNet(specs, wl.head, weights, hp)


def region_codes(zs):
    """NITRO-ReLU segment per element as the library stores it: 0 identity, 1 leaky, 2 saturated."""
    zs = np.asarray(zs)
    return np.where((zs >= 0) & (zs <= 127), 0, np.where((zs < 0) & (zs >= -127), 1, 2))


def pooled_codes(zs, idx):
    """Per pooled element: winning window index | the winner's segment << 2."""
    N_, H, W, C = zs.shape
    v = np.asarray(zs).reshape(N_, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
    win = np.take_along_axis(v.reshape(N_, H // 2, W // 2, 4, C), idx[:, :, :, None, :], axis=3)[..., 0, :]
    return idx + 4 * region_codes(win)


def check_training(ctx, wl, steps, nm, om):
    """nitro_train_step against OracleNet.train_step: after every step, every tensor the
    iteration leaves in its workspace (block outputs, inner activations, region codes, yhat, e,
    every weight gradient, the output layer's yhat, e and weight gradient) and every weight."""
    print("training case", wl.name, "batch", wl.batch, "steps", steps, "mode", nm, flush=True)
    dr = WL.draw_workload(wl, O.kaiming_bound, steps=steps)
    ref = oracle_net(wl, dr.weights, om)
    net = runner.GpuNet(wl, dr.weights, nm, ctx=ctx)

    def same(t, a, what):
        assert np.array_equal(host(t), np.asarray(a)), what

    for s, (x, y) in enumerate(dr.batches):
        st = ref.train_step(x, y)
        net.step(dev(x), dev(y))
        ctx.sync()
        for b, rec in enumerate(st.blocks):
            v = net.view(b)
            tag = "step %d block %d " % (s, b)
            same(v["a_out"], rec.out, tag + "output")
            J = len(rec.layers)
            for j, ly in enumerate(rec.layers):
                if j < J - 1:
                    same(v["act"][j], ly.a, tag + "activation %d" % j)
                    same(v["code"][j], region_codes(ly.zs), tag + "codes %d" % j)
                same(v["dw"][j], rec.dw[j], tag + "dW %d" % j)
            last = rec.layers[-1]
            code = (pooled_codes(last.zs, rec.pool_idx) if rec.pool_idx is not None
                    else region_codes(last.zs))
            if rec.keep is not None:       # a dropped output's region reads "saturated"
                code = np.where(rec.keep, code, (code & 3) + 8 if rec.pool_idx is not None else 2)
            same(v["code"][J - 1], code, tag + "codes %d" % (J - 1))
            same(v["yhat"], rec.yhat, tag + "yhat")
            same(v["e"], rec.e, tag + "e")
            same(v["dw_lr"], rec.dw_lr, tag + "dW learning")
        if wl.head:
            hv = net.head_view()
            same(hv["yhat"], st.head_yhat, "step %d head yhat" % s)
            same(hv["e"], st.head_e, "step %d head e" % s)
            same(hv["dw"], st.head_dw, "step %d head dW" % s)
        for k, (wg, wo) in enumerate(zip(net.weights_np(), ref.w)):
            assert np.array_equal(wg, wo), "step %d weight tensor %d" % (s, k)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_tiny_cnn(ctx, modes):
    check_training(ctx, WL.TINY_CNN, 10, *modes)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_mlp(ctx, modes):
    check_training(ctx, WL.MLP, 10, *modes)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_small_cnn(ctx, modes):
    check_training(ctx, WL.SMALL_CNN, 10, *modes)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_vgg_reduced_batch(ctx, modes):
    check_training(ctx, WL.scaled(WL.VGG_CNN, 4), 10, *modes)


@pytest.mark.parametrize("wl,steps", [(WL.scaled(WL.VGG8B, 2), 3), (WL.scaled(WL.VGG11B, 2), 2),
                                      (WL.MLP3, 10), (WL.scaled(WL.MLP4, 8), 3)],
                         ids=["vgg8b_b2", "vgg11b_b2", "mlp3_b64", "mlp4_b8"])
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_paper_nets(ctx, wl, steps, modes):
    """The paper's architectures (Tab. 1, Tab. 6 hyper-parameters): learning layers on the
    block outputs max-pooled to 4096 features, a linear block after the conv blocks, the
    output layer; every workspace tensor and weight after every step."""
    check_training(ctx, wl, steps, *modes)


@pytest.mark.parametrize("wl", [
    dataclasses.replace(WL.scaled(WL.SMALL_CNN, 8), dropout_conv_ppm=300000, dropout_seed=12345),
    dataclasses.replace(WL.MLP, dropout_lin_ppm=500000, dropout_seed=7),
    dataclasses.replace(WL.scaled(WL.VGG8B, 2), dropout_conv_ppm=100000, dropout_lin_ppm=150000,
                        dropout_seed=99),
    dataclasses.replace(WL.scaled(WL.TINY_CNN, 4), dropout_conv_ppm=1000000)],
    ids=["small_cnn_pc30", "mlp_pl50", "vgg8b_pc10_pl15", "tiny_cnn_pc100"])
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_train_dropout(ctx, wl, modes):
    """Dropout of block outputs with the Philox4x64-10 masks (conv and linear blocks, pooled and
    unpooled, rates up to 1): every workspace tensor and weight after every step."""
    check_training(ctx, wl, 4, *modes)


@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_conv_stress_reduced_batch(ctx, modes):
    """The single conv layer at batch 2, ten repeats with IntegerSGD (through
    nitro_block_sgd_step) between them: every tensor of every repeat."""
    wl = WL.scaled(WL.CONV_STRESS, 2)
    print("stress case batch", wl.batch, "mode", modes[0], flush=True)
    dr = WL.draw_workload(wl, O.kaiming_bound)
    ref = oracle_net(wl, dr.weights, modes[1])
    st = runner.GpuConvStress(wl, dr.weights[0], modes[0], ctx=ctx)
    x, _ = dr.batches[0]
    xd, dd = dev(x), dev(dr.delta)
    g = torch.empty(dr.delta.shape, dtype=torch.int32, device=DEV)
    for r in range(10):
        rec = ref.stress_repeat(x, dr.delta)
        # (odd repeats: g untapped, passed to the weight-gradient preparation in 16 bits)
        st.repeat(xd, dd, taps={"g": [g]} if r % 2 == 0 else None)
        ctx.sync()
        assert np.array_equal(host(st.a), rec.out), "repeat %d output" % r
        if r % 2 == 0:
            assert np.array_equal(host(g), rec.g[0]), "repeat %d g" % r
        assert np.array_equal(host(st.dw), rec.dw[0]), "repeat %d dW" % r
        assert np.array_equal(host(st.dx), rec.dx), "repeat %d dx" % r
        assert np.array_equal(host(st.w), ref.w[0]), "repeat %d W" % r


@pytest.mark.parametrize("af", [0, 640])
def test_block_sgd_step(ctx, af):
    """nitro_block_sgd_step: forward layers with AF * gamma (AF = 2^6 G, or given), learning
    layer with gamma, against the oracle's IntegerSGD on every tensor."""
    rng = np.random.default_rng(21)
    G, d = 10, 48
    desc = N.block_desc(2, 4, 4, [N.layer(N.CONV3X3, 8, 12), N.layer(N.CONV3X3, 12, 12)], True,
                        G, 10)
    ws = [rand(rng, (12, 3, 3, 8), -(1 << 20), 1 << 20, np.int32),
          rand(rng, (12, 3, 3, 12), -(1 << 20), 1 << 20, np.int32)]
    wlr = rand(rng, (G, d), -(1 << 20), 1 << 20, np.int32)
    dws = [rand(rng, w.shape, -(1 << 40), 1 << 40, np.int64) for w in ws]
    dwlr = rand(rng, (G, d), -(1 << 30), 1 << 30, np.int64)
    gamma, lam_fw, lam_lr = 512, 25, 3
    wd = [dev(w) for w in ws]
    wlrd = dev(wlr)
    ctx.block_sgd_step(desc, wd, wlrd, [dev(a) for a in dws], dev(dwlr),
                       N.hparams(gamma, lam_fw, lam_lr, af=af))
    ctx.sync()
    gfw = (af or (1 << 6) * G) * gamma
    for w, dw, wg in zip(ws, dws, wd):
        assert np.array_equal(host(wg), O.integer_sgd(w, dw, gfw, lam_fw))
    assert np.array_equal(host(wlrd), O.integer_sgd(wlr, dwlr, gamma, lam_lr))


def test_deterministic(ctx):
    wl = WL.scaled(WL.SMALL_CNN, 8)
    dr = WL.draw_workload(wl, O.kaiming_bound, steps=3)
    outs = []
    for _ in range(2):
        net = runner.GpuNet(wl, dr.weights, ctx=ctx)
        for x, y in dr.batches:
            net.step(dev(x), dev(y))
        ctx.sync()
        outs.append(net.weights_np())
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("naux", [0, 1, 2])
def test_train_step_aux_streams(ctx, naux):
    """The blocks' local training on 0, 1 or 2 auxiliary streams gives the weights of the
    default 3 (nitro_set_aux_streams), step after step."""
    wl = WL.scaled(WL.VGG_CNN, 4)
    dr = WL.draw_workload(wl, O.kaiming_bound, steps=3)
    outs = []
    for n in (3, naux):
        ctx.set_aux_streams(n)
        try:
            net = runner.GpuNet(wl, dr.weights, ctx=ctx)
            for x, y in dr.batches:
                net.step(dev(x), dev(y))
            ctx.sync()
            outs.append(net.weights_np())
        finally:
            ctx.set_aux_streams(3)
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("feed", ["copy", "resident", "prepared"])
@pytest.mark.parametrize("wl,nbuf", [(WL.scaled(WL.SMALL_CNN, 16), 18), (WL.scaled(WL.VGG_CNN, 8), 4)],
                         ids=["small_cnn_b16", "vgg_b8"])
def test_train_step_graph_matches_eager(wl, nbuf, feed):
    """nitro_train_step_graph replays captured iterations: after every replay (with eager torch
    work and host syncs in between) its weights and block outputs equal the eager path's, which
    the oracle-parity tests pin. The batch changes by writing into the captured buffers (copy),
    or by passing one of nbuf resident buffer sets, each replayed from a graph of its own
    (resident; on the small network more sets than the context keeps graphs for, so that graphs
    are replaced and captured again), or so with every set's graph prepared first
    (nitro_train_step_graph_prepare, which must leave the weights untouched)."""
    import torch
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        gctx = N.Context(0, stream=stream)
        ectx = N.Context(0, stream=stream)
        dr = WL.draw_workload(wl, O.kaiming_bound, steps=4)
        eager = runner.GpuNet(wl, dr.weights, ctx=ectx)
        graph = runner.GpuNet(wl, dr.weights, ctx=gctx)
        xb = torch.empty_like(dev(dr.batches[0][0]))
        yb = torch.empty_like(dev(dr.batches[0][1]))
        bufs = [(dev(dr.batches[k % 4][0]), dev(dr.batches[k % 4][1])) for k in range(nbuf)]
        steps = 8 if feed == "copy" else 2 * nbuf
        if feed == "prepared":
            w_init = graph.weights_np()
            for xd, yd in bufs:
                graph.prepare_graph(xd, yd)
            torch.cuda.synchronize()
            gctx.sync()
            for a, b in zip(w_init, graph.weights_np()):
                assert np.array_equal(a, b), "preparing a graph changed the weights"
        for s in range(steps):
            k = s % nbuf if feed != "copy" else s % 4
            print("graph replay", wl.name, feed, "step", s, "batch", k % 4, flush=True)
            xd, yd = bufs[k] if feed != "copy" else (dev(dr.batches[k][0]), dev(dr.batches[k][1]))
            eager.step(xd, yd)
            if feed != "copy":
                graph.step_graph(xd, yd)
            else:
                xb.copy_(xd)
                yb.copy_(yd)
                graph.step_graph(xb, yb)
            junk = torch.ones(1 << 16, device="cuda", dtype=torch.int32).cumsum(0)   # eager work
            torch.cuda.synchronize()
            gctx.sync()
            ectx.sync()
            for a, b in zip(eager.weights_np(), graph.weights_np()):
                assert np.array_equal(a, b), "step %d weights" % s
            for b in range(len(wl.blocks)):
                assert torch.equal(eager.block_output(b), graph.block_output(b)), "step %d block %d" % (s, b)
            del junk
        gctx.close()
        ectx.close()


@pytest.mark.parametrize("wl,steps", [(WL.TINY_CNN, 2), (WL.MLP, 3), (WL.SMALL_CNN, 2),
                                      (WL.scaled(WL.VGG_CNN, 8), 2), (WL.scaled(WL.VGG8B, 4), 1),
                                      (WL.scaled(WL.MLP4, 16), 1)],
                         ids=["tiny_cnn", "mlp", "small_cnn", "vgg_b8", "vgg8b_b4", "mlp4_b16"])
@pytest.mark.parametrize("modes", MODES, ids=["floor", "trunc"])
def test_infer(ctx, wl, steps, modes):
    """nitro_net_infer against the oracle's inference (forward, prediction, first-maximum
    argmax) on an unseen batch, before and after some training steps (the predictions are
    small integers, so ties between classes occur and the first-maximum rule is exercised)."""
    print("inference case", wl.name, "batch", wl.batch, "mode", modes[0], flush=True)
    dr = WL.draw_workload(wl, O.kaiming_bound, steps=steps + 1)
    ref = oracle_net(wl, dr.weights, modes[1])
    net = runner.GpuNet(wl, dr.weights, modes[0], ctx=ctx)
    xt, _ = dr.batches[-1]
    ties = 0
    for s in range(steps + 1):
        yh, pr = net.infer(dev(xt))
        ryh, rpr = ref.infer(xt)
        ctx.sync()
        assert np.array_equal(host(yh), ryh), "step %d yhat" % s
        assert np.array_equal(host(pr), rpr), "step %d prediction" % s
        ties += int(np.sum(np.sum(ryh == ryh.max(axis=1, keepdims=True), axis=1) > 1))
        if s < steps:
            x, y = dr.batches[s]
            ref.train_step(x, y)
            net.step(dev(x), dev(y))
    print("rows with tied maxima:", ties, flush=True)
