"""Write the full-size expected results of the benchmark-sized workloads as digests.

Runs only the CPU oracle (``oracle/``) on the seeded draws of ``paper_2407_11698_amd/workloads.py``
and stores, for every step, the SHA-256 of every tensor the oracle computes, in the dtype the
library stores it in (little-endian, C order), together with a few seeded sample values of each
tensor so that a mismatch can be located. The GPU tests compare the library's tensors with these
digests after every step.

  * VGG-style CNN, batch 256, 100 classes, ten training iterations (floor rounding):
    per block the inner activations, the region codes, the block output and its pooled codes,
    yhat, e, the learning-layer weight gradient, delta^fw at the block output, the gradient at
    every layer's pre-activation and every weight gradient; then every weight after the update.
  * single conv layer 256 -> 256 on 256x256x32x32, twenty repeats with IntegerSGD between them:
    the activations, region codes, the gradient at the pre-activation, the weight gradient, the
    int64 input gradient and the weights after the update;
  * the paper's architectures VGG8B, VGG11B, MLP 3 and MLP 4 at their batch of 64, three training
    iterations each (learning-layer pooling, dropout), through the whole-iteration call: every
    tensor but delta^fw and the pre-activation gradients, and the output layer's tensors.

Usage: ``python tests/golden/make_digests.py [vgg|stress|paper|all]`` (the single conv layer takes
about half an hour on 8 cores).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import oracle as O                         # noqa: E402
from paper_2407_11698_amd import workloads as WL       # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLES = 24

DTYPES = {"int8": np.int8, "uint8": np.uint8, "int32": np.int32, "int64": np.int64}


def as_dtype(a, dtype: str) -> np.ndarray:
    """The tensor in the library's storage dtype (its values must fit)."""
    a = np.asarray(a)
    info = np.iinfo(DTYPES[dtype])
    if a.size:
        assert info.min <= a.min() and a.max() <= info.max, (dtype, a.min(), a.max())
    return np.ascontiguousarray(a.astype(DTYPES[dtype]))


def sample_positions(key: str, size: int) -> np.ndarray:
    """Seeded flat positions for a tensor's sample values (the same on both sides)."""
    seed = int.from_bytes(hashlib.sha256(key.encode()).digest()[:8], "little")
    return np.random.default_rng(seed).integers(0, size, SAMPLES)


def record(a, dtype: str, key: str) -> dict:
    t = as_dtype(a, dtype)
    flat = t.reshape(-1)
    pos = sample_positions(key, flat.size) if flat.size else np.zeros(0, np.int64)
    return {"dtype": dtype, "shape": list(t.shape),
            "sha256": hashlib.sha256(t.tobytes()).hexdigest(),
            "sample": [[int(p), int(flat[p])] for p in pos]}


def region_codes(zs) -> np.ndarray:
    """NITRO-ReLU segment of each rescaled pre-activation, as the library stores it: 0 identity
    (0 <= z* <= 127), 1 leaky (-127 <= z* < 0), 2 saturated."""
    zs = np.asarray(zs)
    return np.where((zs >= 0) & (zs <= 127), 0, np.where((zs < 0) & (zs >= -127), 1, 2))


def pooled_codes(zs, idx) -> np.ndarray:
    """Per pooled element: the winning window index | the winner's segment << 2."""
    N, H, W, C = zs.shape
    v = np.asarray(zs).reshape(N, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
    v = v.reshape(N, H // 2, W // 2, 4, C)
    win = np.take_along_axis(v, idx[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return idx + 4 * region_codes(win)


def train_digests(wl, steps: int, taps: bool) -> dict:
    """Every tensor of `steps` training iterations of workload `wl`: per block the inner
    activations and region codes, the block output and its codes (dropped outputs, when the
    workload has dropout, read "saturated"), yhat, e and every weight gradient; with `taps` also
    delta^fw and the gradient at every layer's pre-activation; the output layer's yhat, e and
    weight gradient; every weight after the update."""
    dr = WL.draw_workload(wl, O.kaiming_bound, steps=steps)
    hp = O.Hyper(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr, wl.alpha_inv, wl.n_classes,
                 d_lr=wl.d_lr, dropout_conv_ppm=wl.dropout_conv_ppm,
                 dropout_lin_ppm=wl.dropout_lin_ppm, dropout_seed=wl.dropout_seed)
    net = O.OracleNet([(len(b.layers), b.maxpool, b.learning) for b in wl.blocks], wl.head,
                      dr.weights, hp)
    out = {"workload": wl.name, "batch": wl.batch, "rounding": "floor", "steps": []}
    for s, (x, y) in enumerate(dr.batches):
        t0 = time.time()
        st = net.train_step(x, y)
        rec = {}

        def put(name, a, dtype):
            rec[name] = record(a, dtype, "%s/%d/%s" % (wl.name, s, name))

        for b, blk in enumerate(st.blocks):
            J = len(blk.layers)
            for j, ly in enumerate(blk.layers):
                if j < J - 1:
                    put("b%d.act%d" % (b, j), ly.a, "int8")
                    put("b%d.code%d" % (b, j), region_codes(ly.zs), "uint8")
                if taps:
                    put("b%d.g%d" % (b, j), blk.g[j], "int32")
                put("b%d.dw%d" % (b, j), blk.dw[j], "int64")
            put("b%d.out" % b, blk.out, "int8")
            pooled = blk.pool_idx is not None
            code = (pooled_codes(blk.layers[-1].zs, blk.pool_idx) if pooled
                    else region_codes(blk.layers[-1].zs))
            if blk.keep is not None:
                code = np.where(blk.keep, code, (code & 3) + 8 if pooled else 2)
            put("b%d.code%d" % (b, J - 1), code, "uint8")
            put("b%d.yhat" % b, blk.yhat, "int32")
            put("b%d.e" % b, blk.e, "int32")
            put("b%d.dw_lr" % b, blk.dw_lr, "int64")
            if taps:
                put("b%d.delta" % b, blk.delta_fw.reshape(blk.f.shape), "int32")
        if wl.head:
            put("head.yhat", st.head_yhat, "int32")
            put("head.e", st.head_e, "int32")
            put("head.dw", st.head_dw, "int64")
        for k, w in enumerate(net.w):
            put("w%d" % k, w, "int32")
        out["steps"].append(rec)
        print("%s step %d: %.1f s" % (wl.name, s, time.time() - t0), flush=True)
    return out


def vgg_digests(steps: int = 10) -> dict:
    return train_digests(WL.VGG_CNN, steps, taps=True)


def stress_digests(repeats: int = 20) -> dict:
    wl = WL.CONV_STRESS
    dr = WL.draw_workload(wl, O.kaiming_bound)
    hp = O.Hyper(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr, wl.alpha_inv, 0,
                 af_classes=wl.af_classes)
    net = O.OracleNet([(1, False, False)], False, dr.weights, hp)
    x, _ = dr.batches[0]
    out = {"workload": wl.name, "batch": wl.batch, "rounding": "floor", "steps": []}
    for r in range(repeats):
        t0 = time.time()
        blk = net.stress_repeat(x, dr.delta)
        rec = {}

        def put(name, a, dtype):
            rec[name] = record(a, dtype, "%s/%d/%s" % (wl.name, r, name))

        put("a", blk.out, "int8")
        put("code", region_codes(blk.layers[0].zs), "uint8")
        put("g", blk.g[0], "int32")
        put("dw", blk.dw[0], "int64")
        put("dx", blk.dx, "int64")
        put("w", net.w[0], "int32")
        out["steps"].append(rec)
        del blk
        print("stress repeat %d: %.1f s" % (r, time.time() - t0), flush=True)
    return out


def main():
    which = sys.argv[1] if len(sys.argv) > 1 else "all"
    jobs = []
    if which in ("vgg", "all"):
        jobs.append(("digests_vgg_cnn_b256.json", vgg_digests))
    if which in ("stress", "all"):
        jobs.append(("digests_conv_stress.json", stress_digests))
    if which in ("paper", "all"):
        for wl in WL.PAPER_NETS:
            jobs.append(("digests_%s.json" % wl.name, lambda wl=wl: train_digests(wl, 3, taps=False)))
    for name, fn in jobs:
        d = fn()
        with open(os.path.join(HERE, name), "w") as f:
            json.dump(d, f, separators=(",", ":"))
        print("wrote", name, flush=True)


if __name__ == "__main__":
    main()
