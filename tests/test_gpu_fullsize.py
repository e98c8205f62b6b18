"""Parity at full size, in the configuration bench.py times: every tensor after every step.

The oracle's results for the benchmark-sized workloads are stored as per-step SHA-256 digests of
every tensor (``tests/golden/make_digests.py``, which runs only the oracle): the VGG-style CNN at
batch 256 over its ten training iterations, the single 256 -> 256 conv layer on 256x256x32x32
over its twenty repeats with IntegerSGD between them, and the paper's VGG8B, VGG11B, MLP 3 and
MLP 4 at batch 64 over three iterations. Each GPU tensor is hashed in
its storage dtype and must match; on a mismatch the stored sample values name the positions that
differ.

The VGG iteration is run twice in lockstep: through nitro_train_step (what the benchmark calls;
its workspace views give the activations, region codes, yhat, e and every weight gradient) and
through the block-level calls with every tap (which add delta^fw and the gradient at each layer's
pre-activation). Both must produce the oracle's weights after every step."""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

from paper_2407_11698_amd import nitro as N
from paper_2407_11698_amd import runner
from paper_2407_11698_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)
GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
DTYPES = {"int8": torch.int8, "uint8": torch.uint8, "int32": torch.int32, "int64": torch.int64}


@pytest.fixture(scope="module")
def ctx():
    c = N.Context(0)
    yield c
    c.close()


def load_digests(name):
    path = os.path.join(GOLD, name)
    if not os.path.exists(path):
        pytest.fail("%s is missing: run tests/golden/make_digests.py" % path)
    with open(path) as f:
        return json.load(f)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def check(exp: dict, name: str, t: torch.Tensor, where: str):
    """The tensor's digest (in the stored dtype) against the oracle's; on a mismatch, report the
    sample positions that differ."""
    e = exp[name]
    assert t.dtype == DTYPES[e["dtype"]], (where, name, t.dtype)
    assert list(t.shape) == e["shape"], (where, name, list(t.shape), e["shape"])
    a = t.contiguous().cpu().numpy()
    if hashlib.sha256(a.tobytes()).hexdigest() == e["sha256"]:
        return
    flat = a.reshape(-1)
    bad = [(p, v, int(flat[p])) for p, v in e["sample"] if int(flat[p]) != v]
    pytest.fail("%s %s differs from the oracle; sampled (position, oracle, gpu) mismatches: %s"
                % (where, name, bad[:8] or "none among the samples"))


class BlockLevelNet:
    """nitro_train_step spelled out with the block-level calls, keeping every tap."""

    def __init__(self, ctx, wl, weights):
        self.ctx, self.wl = ctx, wl
        self.descs = runner.block_descs(wl)
        self.hp = N.hparams(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr)
        self.w = [dev(w) for w in weights]
        self.blocks = []
        k = 0
        for b, (desc, blk, (inp, out)) in enumerate(zip(self.descs, wl.blocks, wl.block_shapes())):
            J = len(blk.layers)
            ws = self.w[k:k + J]
            wlr = self.w[k + J]
            k += J + 1
            c, h, w = out
            _, h0, w0 = inp
            taps = {"yhat": torch.empty((wl.batch, wl.n_classes), dtype=torch.int32, device=DEV),
                    "e": torch.empty((wl.batch, wl.n_classes), dtype=torch.int32, device=DEV),
                    "delta": torch.empty((wl.batch, h, w, c), dtype=torch.int32, device=DEV),
                    "g": [torch.empty((wl.batch, h0, w0, ly.c_out), dtype=torch.int32, device=DEV)
                          for ly in blk.layers]}
            self.blocks.append(dict(
                desc=desc, ws=ws, wlr=wlr, J=J, hw=(h0, w0), chans=[ly.c_out for ly in blk.layers],
                state=torch.empty(N.block_query(desc), dtype=torch.uint8, device=DEV),
                a_out=torch.empty((wl.batch, h, w, c), dtype=torch.int8, device=DEV),
                dws=[torch.empty(t.shape, dtype=torch.int64, device=DEV) for t in ws],
                dw_lr=torch.empty((wl.n_classes, c * h * w), dtype=torch.int64, device=DEV),
                taps=taps))

    def step(self, x, y):
        cur = x
        for B in self.blocks:
            self.ctx.block_forward(B["desc"], B["ws"], cur, B["a_out"], B["state"])
            B["x"] = cur
            cur = B["a_out"]
        for B in self.blocks:
            self.ctx.block_backward(B["desc"], B["ws"], B["wlr"], B["x"], B["a_out"], y, None,
                                    B["state"], B["dws"], B["dw_lr"], B["taps"])
        for B in self.blocks:
            self.ctx.block_sgd_step(B["desc"], B["ws"], B["wlr"], B["dws"], B["dw_lr"], self.hp)
        self.ctx.sync()

    def saved(self, B, j, what):
        """Layer j's saved int8 activations ("act") or region codes ("code") in the state."""
        act, code = N.block_saved(B["desc"], B["state"], j)
        n = self.wl.batch
        h, w = B["hw"]
        pooled = j == B["J"] - 1 and B["desc"].maxpool
        shape = (n, h // 2, w // 2, B["chans"][j]) if pooled else (n, h, w, B["chans"][j])
        ptr, dt = (act, torch.int8) if what == "act" else (code, torch.uint8)
        off = ptr - B["state"].data_ptr()
        return B["state"][off:off + int(np.prod(shape))].view(dt).view(shape)


def test_vgg_full_batch_every_tensor(ctx):
    """The benchmark workload (batch 256, 100 classes), all ten steps of its trajectory, every
    tensor of both the whole-iteration call and the block-level calls."""
    wl = WL.VGG_CNN
    dg = load_digests("digests_vgg_cnn_b256.json")
    assert dg["workload"] == wl.name and dg["batch"] == wl.batch
    print("full-size case", wl.name, flush=True)
    dr = WL.draw_workload(wl, runner.kaiming_bound, steps=len(dg["steps"]))
    blk_net = BlockLevelNet(ctx, wl, dr.weights)
    net = runner.GpuNet(wl, dr.weights, ctx=ctx)
    for s, ((x, y), exp) in enumerate(zip(dr.batches, dg["steps"])):
        print("step", s, flush=True)
        xd, yd = dev(x), dev(y)
        blk_net.step(xd, yd)
        net.step(xd, yd)
        ctx.sync()
        for b, B in enumerate(blk_net.blocks):
            v = net.view(b)
            for path, src in (("train_step", v), ("block calls", None)):
                where = "step %d (%s)" % (s, path)
                for j in range(B["J"]):
                    if j < B["J"] - 1:
                        act = v["act"][j] if src else blk_net.saved(B, j, "act")
                        check(exp, "b%d.act%d" % (b, j), act, where)
                    code = v["code"][j] if src else blk_net.saved(B, j, "code")
                    check(exp, "b%d.code%d" % (b, j), code, where)
                    check(exp, "b%d.dw%d" % (b, j), v["dw"][j] if src else B["dws"][j], where)
                    if not src:
                        check(exp, "b%d.g%d" % (b, j), B["taps"]["g"][j], where)
                check(exp, "b%d.out" % b, v["a_out"] if src else B["a_out"], where)
                check(exp, "b%d.yhat" % b, v["yhat"] if src else B["taps"]["yhat"], where)
                check(exp, "b%d.e" % b, v["e"] if src else B["taps"]["e"], where)
                check(exp, "b%d.dw_lr" % b, v["dw_lr"] if src else B["dw_lr"], where)
                if not src:
                    check(exp, "b%d.delta" % b, B["taps"]["delta"], where)
        for k in range(len(net.w)):
            check(exp, "w%d" % k, net.w[k], "step %d (train_step)" % s)
            check(exp, "w%d" % k, blk_net.w[k], "step %d (block calls)" % s)


def test_conv_stress_full_size_twenty_repeats(ctx):
    """256x256x32x32, conv 256 -> 256, fixed activations and error signal, twenty cumulative
    repeats with IntegerSGD between them (the weights leave int8 after the first). g is tapped on
    even repeats only: untapped, the library passes it to the weight-gradient preparation in 16
    bits (as in the bench's repeats)."""
    wl = WL.CONV_STRESS
    dg = load_digests("digests_conv_stress.json")
    assert dg["workload"] == wl.name and dg["batch"] == wl.batch
    print("full-size case", wl.name, flush=True)
    dr = WL.draw_workload(wl, runner.kaiming_bound)
    x, _ = dr.batches[0]
    st = runner.GpuConvStress(wl, dr.weights[0], ctx=ctx)
    g = torch.empty(dr.delta.shape, dtype=torch.int32, device=DEV)
    xd, dd = dev(x), dev(dr.delta)
    _, code_ptr = N.block_saved(st.desc, st.state, 0)
    off = code_ptr - st.state.data_ptr()
    code = st.state[off:off + st.a.numel()].view(st.a.shape)
    for r, exp in enumerate(dg["steps"]):
        print("repeat", r, flush=True)
        st.repeat(xd, dd, taps={"g": [g]} if r % 2 == 0 else None)
        ctx.sync()
        where = "repeat %d" % r
        check(exp, "a", st.a, where)
        check(exp, "code", code, where)
        if r % 2 == 0:
            check(exp, "g", g, where)
        check(exp, "dw", st.dw, where)
        check(exp, "dx", st.dx, where)
        check(exp, "w", st.w, where)


@pytest.mark.parametrize("name", [wl.name for wl in WL.PAPER_NETS])
def test_paper_nets_full_batch_every_tensor(ctx, name):
    """The paper's architectures at their batch of 64 (learning-layer pooling to 4096 features,
    dropout where Tab. 6 sets it), three training iterations through nitro_train_step: every
    tensor the iteration leaves in its workspace, the output layer's, and every weight."""
    wl = WL.WORKLOADS[name]
    dg = load_digests("digests_%s.json" % name)
    assert dg["workload"] == wl.name and dg["batch"] == wl.batch
    print("full-size case", wl.name, flush=True)
    dr = WL.draw_workload(wl, runner.kaiming_bound, steps=len(dg["steps"]))
    net = runner.GpuNet(wl, dr.weights, ctx=ctx)
    for s, ((x, y), exp) in enumerate(zip(dr.batches, dg["steps"])):
        print("step", s, flush=True)
        net.step(dev(x), dev(y))
        ctx.sync()
        where = "step %d" % s
        for b, blk in enumerate(wl.blocks):
            v = net.view(b)
            J = len(blk.layers)
            for j in range(J):
                if j < J - 1:
                    check(exp, "b%d.act%d" % (b, j), v["act"][j], where)
                check(exp, "b%d.code%d" % (b, j), v["code"][j], where)
                check(exp, "b%d.dw%d" % (b, j), v["dw"][j], where)
            check(exp, "b%d.out" % b, v["a_out"], where)
            check(exp, "b%d.yhat" % b, v["yhat"], where)
            check(exp, "b%d.e" % b, v["e"], where)
            check(exp, "b%d.dw_lr" % b, v["dw_lr"], where)
        hv = net.head_view()
        check(exp, "head.yhat", hv["yhat"], where)
        check(exp, "head.e", hv["e"], where)
        check(exp, "head.dw", hv["dw"], where)
        for k in range(len(net.w)):
            check(exp, "w%d" % k, net.w[k], where)
