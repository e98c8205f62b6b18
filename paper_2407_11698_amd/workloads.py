"""Synthetic workloads shaped like the paper's experiments, and their seeded input generators.

This module holds configuration and random draws only: no arithmetic of the method lives here
(no scaling factors, no NITRO-ReLU, no IntegerSGD, no initialisation bound). Both the product
path and the test-side checker draw their inputs from here, so that they see identical arrays.

Shapes follow the datasets named in the experimental section (28x28 grey images with 10 classes,
32x32 RGB images with 10 or 100 classes) and the architectures of Tab. 1 (3x3 convolutions,
stride 1, padding 1; 2x2 max-pool, stride 2). The datasets themselves are not used: every input
is drawn uniformly from the int8 operational range [-127, 127].

Layouts of the generated host arrays:
  * images: drawn as NCHW, returned as NHWC int8 (channels innermost);
  * MLP inputs: [N, D] int8;
  * conv weights: drawn as [C_out][C_in][3][3], returned as KRSC [C_out][3][3][C_in] int32;
  * linear / learning / head weights: [out][in] int32, the input index in (h, w, c) order;
  * labels: [N] int32 in [0, G).

Draw order for one workload (one PCG64 stream, ``numpy.random.default_rng(seed)``):
  1. weights, block by block: the forward layers in order, then that block's learning layer;
     then the output head;
  2. for each step s = 0, 1, ...: the input batch x_s, then the labels y_s.
The single-layer stress workload draws its weight, then the activations a, then the error
signal delta, once (the repeats reuse them).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Conv3x3:
    """IntConv2D, 3x3 kernel, stride 1, zero padding 1, no bias (Tab. 1 caption)."""
    c_in: int
    c_out: int

    @property
    def fan_in(self) -> int:
        return 9 * self.c_in


@dataclass(frozen=True)
class Linear:
    """IntLinear without bias (section 3.2.1)."""
    d_in: int
    d_out: int

    @property
    def fan_in(self) -> int:
        return self.d_in


@dataclass(frozen=True)
class Init:
    """How a weight tensor is drawn: ``uniform`` with a literal bound, or ``kaiming``.

    For ``kaiming`` the bound is a function of ``fan_in`` defined in section 3.3.1; the caller
    computes it and passes it to :func:`draw_weights`.
    """
    kind: str            # "uniform" | "kaiming"
    bound: int = 0       # used when kind == "uniform"


@dataclass(frozen=True)
class Block:
    """One integer local-loss block (section 3.2): forward layers, optional 2x2 max-pool after the
    last NITRO-ReLU, and an optional learning layer (IntLinear d -> G) on the block output."""
    layers: Tuple[object, ...]
    maxpool: bool
    learning: bool
    init: Init = Init("kaiming")


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    in_shape: Tuple[int, ...]          # (C, H, W) for images, (D,) for MLP inputs
    blocks: Tuple[Block, ...]
    n_classes: int                     # G; 0 for the single-layer stress case
    head: bool                         # an output layer IntLinear(d_L -> G)
    gamma_inv: int                     # gamma_inv of the learning layers (Tab. 6 caption)
    lambda_inv_fw: int
    lambda_inv_lr: int
    alpha_inv: int
    steps: int
    seed: int = 0
    head_init: Init = Init("kaiming")
    af_classes: int = 0                # G used for the amplification factor when n_classes == 0
    delta_bound: int = 0               # stress case: |delta| <= delta_bound at the ReLU output
    d_lr: int = 0                      # learning-layer input size of conv blocks (d^lr, Tab. 6);
    #                                    0: the learning layer reads the block output
    dropout_conv_ppm: int = 0          # dropout rates p_c, p_l of Tab. 6, parts per million
    dropout_lin_ppm: int = 0
    dropout_seed: int = 0              # key of the dropout generator

    # ---- derived shapes (bookkeeping only) ----
    @property
    def is_image(self) -> bool:
        return len(self.in_shape) == 3

    def block_shapes(self):
        """Per block: (input shape, output shape after pool) in per-sample NHWC / [D] terms."""
        shapes = []
        cur = tuple(self.in_shape)
        for blk in self.blocks:
            if isinstance(blk.layers[0], Conv3x3):
                c, h, w = cur
                for ly in blk.layers:
                    assert ly.c_in == c, (ly, cur)
                    c = ly.c_out
                if blk.maxpool:
                    h, w = h // 2, w // 2
                out = (c, h, w)
            else:
                d = int(np.prod(cur))          # a conv output is read flattened, (h, w, c) order
                for ly in blk.layers:
                    assert ly.d_in == d, (ly, cur)
                    d = ly.d_out
                out = (d,)
            shapes.append((cur, out))
            cur = out
        return shapes

    def learning_window(self, b: int):
        """Window (kh, kw) of block b's learning-layer max-pooling (1, 1: none). Shape
        bookkeeping of the library's d_lr rule: kh and kw are doubled in turn, kh first, while
        c (h / kh)(w / kw) > d_lr and a side can still be halved."""
        _, out = self.block_shapes()[b]
        if len(out) != 3 or not self.d_lr or not self.blocks[b].learning:
            return 1, 1
        c, h, w = out
        kh = kw = 1
        turn_h = True
        while c * (h // kh) * (w // kw) > self.d_lr:
            can_h, can_w = (h // kh) % 2 == 0, (w // kw) % 2 == 0
            if not (can_h or can_w):
                break
            if (turn_h and can_h) or not can_w:
                kh *= 2
            else:
                kw *= 2
            turn_h = not turn_h
        return kh, kw

    def learning_dim(self, b: int) -> int:
        _, out = self.block_shapes()[b]
        kh, kw = self.learning_window(b)
        if len(out) == 3:
            return out[0] * (out[1] // kh) * (out[2] // kw)
        return int(np.prod(out))

    def head_dim(self) -> int:
        """Input size of the output layer: the last block's output, flattened."""
        _, out = self.block_shapes()[-1]
        return int(np.prod(out))


U127 = Init("uniform", 127)

# Tiny CNN, one block: 16x1x28x28, conv 1->16, pool, learning 3136 -> 10.
TINY_CNN = Workload(
    name="tiny_cnn_16x1x28x28", batch=16, in_shape=(1, 28, 28),
    blocks=(Block((Conv3x3(1, 16),), maxpool=True, learning=True, init=U127),),
    n_classes=10, head=False, gamma_inv=512, lambda_inv_fw=30000, lambda_inv_lr=3000,
    alpha_inv=10, steps=10)

# Integer MLP 784-100-50-10 (Tab. 1, MLP 1), batch 64; each hidden layer is a block with its own
# learning layer; the final 50 -> 10 layer is the output head.
MLP = Workload(
    name="mlp_784_100_50_10_b64", batch=64, in_shape=(784,),
    blocks=(Block((Linear(784, 100),), maxpool=False, learning=True),
            Block((Linear(100, 50),), maxpool=False, learning=True)),
    n_classes=10, head=True, gamma_inv=512, lambda_inv_fw=12000, lambda_inv_lr=3000,
    alpha_inv=10, steps=10)

# Small CNN on 3x32x32, batch 64: three one-conv blocks with pool, head 2048 -> 10.
SMALL_CNN = Workload(
    name="small_cnn_3blk_b64", batch=64, in_shape=(3, 32, 32),
    blocks=(Block((Conv3x3(3, 32),), maxpool=True, learning=True),
            Block((Conv3x3(32, 64),), maxpool=True, learning=True),
            Block((Conv3x3(64, 128),), maxpool=True, learning=True)),
    n_classes=10, head=True, gamma_inv=512, lambda_inv_fw=25000, lambda_inv_lr=3000,
    alpha_inv=10, steps=10)

# VGG-style CNN, batch 256, 100 classes: four two-conv blocks with pool and a learning layer.
# gamma_inv is the paper's 512 (tuned at batch 64) times 4: IntegerSGD divides a batch *sum*, so
# at batch 256 the same per-sample step needs a 4x larger divisor; at 512 the weights explode in
# two steps and the third step's gradients leave int32.
VGG_CNN = Workload(
    name="vgg_cnn_4x2conv_b256_c100", batch=256, in_shape=(3, 32, 32),
    blocks=(Block((Conv3x3(3, 64), Conv3x3(64, 64)), maxpool=True, learning=True),
            Block((Conv3x3(64, 128), Conv3x3(128, 128)), maxpool=True, learning=True),
            Block((Conv3x3(128, 256), Conv3x3(256, 256)), maxpool=True, learning=True),
            Block((Conv3x3(256, 512), Conv3x3(512, 512)), maxpool=True, learning=True)),
    n_classes=100, head=False, gamma_inv=2048, lambda_inv_fw=25000, lambda_inv_lr=3000,
    alpha_inv=10, steps=10)

# Single conv-layer stress: 256x256x32x32 int8 activations, conv 256 -> 256, a given int32 error
# signal at the ReLU output; forward + dX + dW + Scaling/ReLU + IntegerSGD, 20 repeats.
CONV_STRESS = Workload(
    name="conv_stress_256x256x32x32", batch=256, in_shape=(256, 32, 32),
    blocks=(Block((Conv3x3(256, 256),), maxpool=False, learning=False, init=U127),),
    n_classes=0, head=False, gamma_inv=512, lambda_inv_fw=25000, lambda_inv_lr=3000,
    alpha_inv=10, steps=20, af_classes=10, delta_bound=1 << 15)

# The paper's own architectures (Tab. 1) with the hyper-parameters of Tab. 6 (batch 64, gamma_inv
# 512, the CIFAR-10 or MNIST row). Every IntConv2D with its NITRO-ReLU (and the MaxPool2D that
# follows it, if any) is one local-loss block; every hidden IntLinear is an integer linear block;
# the last IntLinear is the output layer. Conv blocks' learning layers read the block output
# max-pooled to at most d^lr = 4096 features.
def _vgg(name, convs, lam_fw, lam_lr, p_lin_ppm=0):
    blocks = []
    c = 3
    for co, pool in convs:
        blocks.append(Block((Conv3x3(c, co),), maxpool=pool, learning=True))
        c = co
    blocks.append(Block((Linear(512 * 2 * 2, 1024),), maxpool=False, learning=True))
    return Workload(name=name, batch=64, in_shape=(3, 32, 32), blocks=tuple(blocks), n_classes=10,
                    head=True, gamma_inv=512, lambda_inv_fw=lam_fw, lambda_inv_lr=lam_lr,
                    alpha_inv=10, steps=10, d_lr=4096, dropout_lin_ppm=p_lin_ppm, dropout_seed=1)


VGG8B = _vgg("vgg8b_cifar10_b64",
             [(128, False), (256, True), (256, False), (512, True), (512, True), (512, True)],
             25000, 3000, p_lin_ppm=150000)
VGG11B = _vgg("vgg11b_cifar10_b64",
              [(128, False), (128, False), (128, False), (256, True), (256, False), (512, True),
               (512, False), (512, True), (512, True)], 28000, 4500)
MLP3 = Workload(
    name="mlp3_784_1024x3_10_b64", batch=64, in_shape=(784,),
    blocks=(Block((Linear(784, 1024),), maxpool=False, learning=True),
            Block((Linear(1024, 1024),), maxpool=False, learning=True),
            Block((Linear(1024, 1024),), maxpool=False, learning=True)),
    n_classes=10, head=True, gamma_inv=512, lambda_inv_fw=28000, lambda_inv_lr=5000,
    alpha_inv=10, steps=10)
MLP4 = Workload(
    name="mlp4_1024_3000x3_10_b64", batch=64, in_shape=(1024,),
    blocks=(Block((Linear(1024, 3000),), maxpool=False, learning=True),
            Block((Linear(3000, 3000),), maxpool=False, learning=True),
            Block((Linear(3000, 3000),), maxpool=False, learning=True)),
    n_classes=10, head=True, gamma_inv=512, lambda_inv_fw=19000, lambda_inv_lr=7500,
    alpha_inv=10, steps=10, dropout_lin_ppm=100000, dropout_seed=1)

WORKLOADS = {w.name: w for w in (TINY_CNN, MLP, SMALL_CNN, VGG_CNN, CONV_STRESS, VGG8B, VGG11B,
                                 MLP3, MLP4)}
BY_INDEX = (TINY_CNN, MLP, SMALL_CNN, VGG_CNN, CONV_STRESS)
PAPER_NETS = (VGG8B, VGG11B, MLP3, MLP4)


def scaled(wl: Workload, batch: int) -> Workload:
    """The same workload at another batch size (for bounded samples and small parity cases)."""
    from dataclasses import replace
    return replace(wl, batch=batch)


# --------------------------------------------------------------------------------------------
# seeded draws
# --------------------------------------------------------------------------------------------

def uniform_int(rng: np.random.Generator, shape, lo: int, hi: int) -> np.ndarray:
    """Integers uniform on [lo, hi], both ends included, as int64."""
    return rng.integers(lo, hi, size=shape, endpoint=True, dtype=np.int64)


def weight_tensors(wl: Workload):
    """(kind, layer, init) of every weight tensor in draw order.

    kind is "conv", "linear" (a forward layer), "learning" or "head"."""
    out = []
    for bi, blk in enumerate(wl.blocks):
        for ly in blk.layers:
            out.append(("conv" if isinstance(ly, Conv3x3) else "linear", ly, blk.init))
        if blk.learning:
            out.append(("learning", Linear(wl.learning_dim(bi), wl.n_classes), blk.init))
    if wl.head:
        out.append(("head", Linear(wl.head_dim(), wl.n_classes), wl.head_init))
    return out


def draw_weights(wl: Workload, rng: np.random.Generator, kaiming_bound) -> list:
    """Draw every weight tensor; ``kaiming_bound(fan_in) -> int`` is supplied by the caller."""
    ws = []
    for kind, ly, init in weight_tensors(wl):
        b = init.bound if init.kind == "uniform" else int(kaiming_bound(ly.fan_in))
        if kind == "conv":
            w = uniform_int(rng, (ly.c_out, ly.c_in, 3, 3), -b, b)
            w = np.ascontiguousarray(w.transpose(0, 2, 3, 1))        # -> KRSC
        else:
            w = uniform_int(rng, (ly.d_out, ly.d_in), -b, b)
        ws.append(w.astype(np.int32))
    return ws


def draw_batch(wl: Workload, rng: np.random.Generator):
    """One (x, labels) batch: x int8 NHWC (or [N, D]), labels int32."""
    shape = (wl.batch,) + tuple(wl.in_shape)
    x = uniform_int(rng, shape, -127, 127).astype(np.int8)
    if wl.is_image:
        x = np.ascontiguousarray(x.transpose(0, 2, 3, 1))             # NCHW -> NHWC
    y = rng.integers(0, max(wl.n_classes, 1), size=wl.batch, dtype=np.int64).astype(np.int32)
    return x, y


@dataclass
class Draws:
    weights: list
    batches: list = field(default_factory=list)     # [(x, y)] per step
    delta: Optional[np.ndarray] = None               # stress case only


def draw_workload(wl: Workload, kaiming_bound, steps: Optional[int] = None) -> Draws:
    """All seeded draws of a workload in the documented order."""
    rng = np.random.default_rng(wl.seed)
    ws = draw_weights(wl, rng, kaiming_bound)
    if wl.delta_bound:
        c, h, w = wl.in_shape
        x = uniform_int(rng, (wl.batch, c, h, w), -127, 127).astype(np.int8)
        x = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
        c_out = wl.blocks[0].layers[-1].c_out
        d = uniform_int(rng, (wl.batch, c_out, h, w), -wl.delta_bound, wl.delta_bound)
        d = np.ascontiguousarray(d.transpose(0, 2, 3, 1)).astype(np.int32)
        return Draws(ws, [(x, np.zeros(wl.batch, np.int32))], d)
    n = wl.steps if steps is None else steps
    return Draws(ws, [draw_batch(wl, rng) for _ in range(n)])


# --------------------------------------------------------------------------------------------
# raw image bytes for the integer pre-processing (Appendix A)
# --------------------------------------------------------------------------------------------

# stands in for the CIFAR-10 training images: 50000 x 32 x 32 x 3 unsigned bytes
CIFAR10_BYTES = (50000, 32, 32, 3)


def draw_image_bytes(shape, seed: int = 0) -> np.ndarray:
    """Seeded uint8 'pixels' of the given shape (images first): each value is N(120, 55) plus a
    per-image brightness offset N(0, 30), rounded and clipped to [0, 255] (a skewed, clipped
    distribution like natural images' pixel values)."""
    rng = np.random.default_rng(seed)
    n = shape[0]
    per = int(np.prod(shape[1:]))
    out = np.empty((n, per), np.uint8)
    off = rng.normal(0.0, 30.0, n)
    chunk = max(1, (1 << 24) // per)
    for i in range(0, n, chunk):
        j = min(n, i + chunk)
        v = rng.normal(120.0, 55.0, (j - i, per)) + off[i:j, None]
        out[i:j] = np.clip(np.rint(v), 0, 255).astype(np.uint8)
    return out.reshape(shape)
