"""Host-only checks of the C ABI: the library loads, exports every symbol include/nitro.h declares,
its host-side division and NITRO-ReLU mean agree with the hand-worked pins, and argument
validation rejects bad calls before any device work. No GPU needed."""
import json
import os
import re

import numpy as np
import pytest

from paper_2407_11698_amd import nitro as N
from paper_2407_11698_amd import runner
from paper_2407_11698_amd import workloads as WL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = os.path.join(ROOT, "tests", "golden")


def test_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "nitro.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"^\s*(?:[a-z_0-9]+\s*\**\s+)+\**(nitro_[a-z_0-9]+)\s*\(", hdr, re.M))
    assert "nitro_train_step" in declared and "nitro_block_forward" in declared
    assert declared == set(N.EXPORTS)
    for name in declared:
        assert hasattr(N.LIB, name), name


def test_status_strings():
    for code in (N.OK, N.EINVAL, N.EOVERFLOW, N.ELABEL, N.EHIP, N.ENOMEM, N.EUNSUPPORTED):
        assert N.status_str(code) and N.status_str(code) != "unknown status"


def test_host_division_table():
    with open(os.path.join(GOLD, "division.json")) as f:
        g = json.load(f)
    for z, fl, tr in g["rows"]:
        assert N.host_div(z, g["sf"], N.ROUND_FLOOR) == fl
        assert N.host_div(z, g["sf"], N.ROUND_TRUNC) == tr


def test_host_division_against_python():
    """The reciprocal-multiply division equals Python's floor division (and its truncating
    counterpart) for every divisor the workloads use and for random divisors."""
    rng = np.random.default_rng(0)
    divisors = [1, 2, 3, 4, 5, 7, 10, 20, 512, 2304, 6912, 25600, 73728, 147456, 200704,
                294912, 589824, 802816, 1179648, 4194304, 327680, 3276800, 1536000,
                8192000000, 81920000000, (1 << 62) - 1]
    divisors += [int(v) for v in rng.integers(1, 1 << 62, 40)]
    divisors += [int(v) for v in rng.integers(1, 1 << 20, 40)]
    nums = [0, 1, -1, (1 << 62) - 1, -(1 << 62) + 1]
    nums += [int(v) for v in rng.integers(-(1 << 62) + 1, 1 << 62, 300)]
    nums += [int(v) for v in rng.integers(-5000, 5000, 300)]
    for d in divisors:
        extra = [d, -d, d - 1, -d + 1, d + 1, -d - 1, 3 * d, -3 * d, 3 * d - 1, -3 * d + 1]
        for n in nums + [v for v in extra if abs(v) < (1 << 62)]:
            assert N.host_div(n, d, N.ROUND_FLOOR) == n // d, (n, d)
            t = (abs(n) // d) * (1 if n >= 0 else -1)
            assert N.host_div(n, d, N.ROUND_TRUNC) == t, (n, d)


def test_host_relu_mu_table():
    with open(os.path.join(GOLD, "relu.json")) as f:
        t = json.load(f)["mu_table"]
    for a, fl, tr in zip(t["alpha_inv"], t["floor"], t["trunc"]):
        assert N.host_relu_mu(a, N.ROUND_FLOOR) == fl
        assert N.host_relu_mu(a, N.ROUND_TRUNC) == tr


def test_kaiming_host_helper_table():
    with open(os.path.join(GOLD, "kaiming.json")) as f:
        g = json.load(f)
    assert [runner.kaiming_bound(f) for f in g["fan_in"]] == g["bound"]


def _conv_block(**kw):
    args = dict(n=2, h=8, w=8, layers=[N.layer(N.CONV3X3, 3, 8)], maxpool=True, n_classes=10,
                alpha_inv=10)
    args.update(kw)
    d = N.block_desc(args["n"], args["h"], args["w"], args["layers"], args["maxpool"],
                     args["n_classes"], args["alpha_inv"])
    if "n_layers" in kw:
        d.n_layers = kw["n_layers"]
    return d


def test_block_query_accepts_workloads():
    for wl in WL.BY_INDEX:
        for d in runner.block_descs(wl):
            assert N.block_query(d) > 0


@pytest.mark.parametrize("bad", [
    dict(n=0), dict(alpha_inv=1), dict(alpha_inv=0), dict(h=7),                 # odd for pooling
    dict(layers=[]), dict(n_layers=5),
    dict(layers=[N.layer(N.CONV3X3, 3, 8), N.layer(N.CONV3X3, 4, 8)]),           # broken chain
    dict(layers=[N.layer(N.CONV3X3, 0, 8)]), dict(n_classes=-1),
    dict(layers=[N.layer(N.LINEAR, 3, 8)]),                                     # linear needs h=w=1
    dict(layers=[N.layer(7, 3, 8)]),
])
def test_block_query_rejects(bad):
    with pytest.raises(N.NitroError) as ei:
        N.block_query(_conv_block(**bad))
    assert ei.value.code == N.EINVAL


def test_layer_query_is_the_one_layer_block():
    """nitro_layer_query sizes the one-layer block (no pooling, no learning layer) and
    rejects what nitro_block_query rejects."""
    for ly, h, w in ((N.layer(N.CONV3X3, 256, 256), 32, 32), (N.layer(N.CONV3X3, 3, 16), 7, 5),
                     (N.layer(N.LINEAR, 784, 100), 1, 1)):
        ld = N.layer_desc(8, h, w, ly, 10)
        bd = N.block_desc(8, h, w, [ly], False, 0, 10)
        assert N.layer_query(ld) == N.block_query(bd) > 0
    for bad in (N.layer_desc(0, 8, 8, N.layer(N.CONV3X3, 4, 8), 10),
                N.layer_desc(2, 8, 8, N.layer(N.CONV3X3, 4, 8), 1),
                N.layer_desc(2, 8, 8, N.layer(N.LINEAR, 4, 8), 10),
                N.layer_desc(2, 8, 8, N.layer(N.CONV3X3, 4, 8), 10, round_mode=2)):
        with pytest.raises(N.NitroError) as ei:
            N.layer_query(bad)
        assert ei.value.code == N.EINVAL
    import ctypes
    assert N.LIB.nitro_layer_query(None, ctypes.byref(ctypes.c_size_t(0))) == N.EINVAL
    ld = N.layer_desc(2, 8, 8, N.layer(N.CONV3X3, 4, 8), 10)
    assert N.LIB.nitro_layer_forward(None, ld, None, None, None, None) == N.EINVAL
    assert N.LIB.nitro_layer_backward(None, ld, None, None, None, None, None, None, None,
                                      None) == N.EINVAL


def test_net_query_checks_chaining():
    descs = runner.block_descs(WL.VGG_CNN)
    assert N.net_query(N.net_desc(descs, False)) > 0
    broken = list(descs)
    broken[1], broken[2] = broken[2], broken[1]
    with pytest.raises(N.NitroError):
        N.net_query(N.net_desc(broken, False))


def test_null_context_rejected():
    d = _conv_block()
    assert N.LIB.nitro_block_forward(None, d, N.BlockParams(), None, None, None) == N.EINVAL
    assert N.LIB.nitro_integer_sgd_step(None, None, None, 0, 1, 0, -1, 0) == N.EINVAL
    assert N.LIB.nitro_sync_status(None) == N.EINVAL


def test_noalloc_forward_size_limit():
    """nitro_block_forward_noalloc checks the block against its 64 MiB scratch before anything
    else (no device work, no context needed): a VGG-style block at batch 1024 is rejected with
    NITRO_EUNSUPPORTED, a small block gets as far as the missing context (EINVAL), and so does
    one just under the limit."""
    import ctypes
    bp = N.BlockParams()
    bp.w[0] = bp.w[1] = 1                       # never dereferenced: rejected on the host
    one = ctypes.c_void_p(1)
    big = N.block_desc(1024, 32, 32, [N.layer(N.CONV3X3, 64, 128), N.layer(N.CONV3X3, 128, 128)],
                       False, 0, 10)
    assert N.LIB.nitro_block_forward_noalloc(None, big, bp, one, one) == N.EUNSUPPORTED
    small = N.block_desc(2, 8, 8, [N.layer(N.CONV3X3, 64, 128), N.layer(N.CONV3X3, 128, 128)],
                         True, 0, 10)
    assert N.LIB.nitro_block_forward_noalloc(None, small, bp, one, one) == N.EINVAL
    # 256 x 32 x 32 x 64 twice (inner activations and codes) plus the last layer's pooled codes:
    # about 38 MB, inside the limit
    vgg1 = N.block_desc(256, 32, 32, [N.layer(N.CONV3X3, 3, 64), N.layer(N.CONV3X3, 64, 64)],
                        True, 0, 10)
    assert N.LIB.nitro_block_forward_noalloc(None, vgg1, bp, one, one) == N.EINVAL
    # an MLP block whose max slots end at about 14 MB but whose split-K partials of the MFMA
    # linear forward need 67 MB more: the check counts them (their room sits behind the slots)
    bp.w[2] = 1
    mlp = N.block_desc(2048, 1, 1, [N.layer(N.LINEAR, 784, 1024), N.layer(N.LINEAR, 1024, 1024)],
                       False, 0, 10)
    assert N.LIB.nitro_block_forward_noalloc(None, mlp, bp, one, one) == N.EUNSUPPORTED
    bp.w[1] = None
    assert N.LIB.nitro_block_forward_noalloc(None, small, bp, one, one) == N.EINVAL
