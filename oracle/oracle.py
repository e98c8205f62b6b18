"""CPU oracle for the NITRO-D integer-only training step.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module; the product path (the HIP library and its binding) never does, and shares no
code with it.

Everything is exact integer arithmetic on int64 numpy arrays. The GEMM-shaped contractions run in
plain C (``nitro_oracle.c``, int64 accumulators); the elementwise steps are numpy, written in the
paper's order and notation. Every quantity that the product stores in int32 is checked here to fit
int32 and raises ``OverflowError`` otherwise.

Readings of passages that the paper leaves open (each is a switch or a documented constant):
  * integer division: the paper's floor macro (round toward minus infinity) by default; rounding
    toward zero is the alternative mode (``TRUNC``), applied to every division of the step;
  * the mean of NITRO-ReLU is the floor (or trunc) of the sum of the four segment means over 4;
  * the loss gradient is taken per sample, e = yhat - y (the batch sum happens in the weight
    gradient);
  * the backward of NITRO-ReLU is the derivative of its piecewise map evaluated at the stored
    rescaled pre-activation z*: identity for 0 <= z* <= 127, division by alpha_inv (same rounding
    mode) for -127 <= z* < 0, zero where the map saturates (z* > 127 or z* < -127) (switch:
    ``Hyper.relu_grad_ste`` passes the gradient unchanged on the leaky segment instead);
  * max-pool keeps the first maximum of the 2x2 window in row-major order and routes the whole
    gradient to it;
  * delta^fw is computed with the learning-layer weights from before their update (switch:
    ``Hyper.delta_fw_post_update`` takes them after it, the literal order of section 3.3);
  * every layer's scaling factor uses its own fan-in; learning and output layers are rescaled too
    but have no NITRO-ReLU;
  * eta = gamma * lambda is formed in int64 (an explicit eta may override it);
  * the learning layers of a conv block read its output max-pooled to at most d^lr features
    (``learning_pool_window``: height and width halved in turn, first maximum of the window);
    without d^lr they read the block output itself;
  * a linear block after a conv block reads the conv output flattened in (h, w, c) order.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

FLOOR = 0
TRUNC = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nitro_oracle.c")
_SO = os.path.join(_HERE, "libnitro_oracle.so")

INT32_MIN = -(1 << 31)
INT32_MAX = (1 << 31) - 1


# ---------------------------------------------------------------------------------------------
# the C part
# ---------------------------------------------------------------------------------------------

def build(force: bool = False) -> str:
    """Compile nitro_oracle.c into libnitro_oracle.so (gcc, OpenMP)."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-Wall", _SRC, "-o", tmp])
        os.replace(tmp, _SO)
    return _SO


_lib = None


def _c():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        I = ctypes.c_int
        for name in ("or_conv3x3_fwd", "or_conv3x3_dx", "or_conv3x3_dw"):
            getattr(lib, name).argtypes = [P, P, P, I, I, I, I, I]
            getattr(lib, name).restype = None
        for name in ("or_linear_fwd", "or_linear_dx", "or_linear_dw"):
            getattr(lib, name).argtypes = [P, P, P, I, I, I]
            getattr(lib, name).restype = None
        lib.or_num_threads.restype = I
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_c().or_num_threads())


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def _as(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def conv3x3_fwd(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """IntConv2D (section 3.2.1; 3x3, stride 1, pad 1 per Tab. 1). x int8 NHWC, w KRSC -> int64 NHWC."""
    N, H, W, C = x.shape
    CO = w.shape[0]
    assert w.shape == (CO, 3, 3, C)
    x8 = _as(x, np.int8)
    w32 = _as(w, np.int32)
    z = np.empty((N, H, W, CO), np.int64)
    _c().or_conv3x3_fwd(_ptr(x8), _ptr(w32), _ptr(z), N, H, W, C, CO)
    return z


def conv3x3_dx(g: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Input gradient of IntConv2D (its adjoint). g NHWC (C_out), w KRSC -> int64 NHWC (C_in)."""
    N, H, W, CO = g.shape
    C = w.shape[3]
    assert w.shape == (CO, 3, 3, C)
    g64 = _as(g, np.int64)
    w32 = _as(w, np.int32)
    dx = np.empty((N, H, W, C), np.int64)
    _c().or_conv3x3_dx(_ptr(g64), _ptr(w32), _ptr(dx), N, H, W, C, CO)
    return dx


def conv3x3_dw(g: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Weight gradient of IntConv2D summed over the batch -> int64 KRSC."""
    N, H, W, CO = g.shape
    C = x.shape[3]
    assert x.shape == (N, H, W, C)
    g64 = _as(g, np.int64)
    x8 = _as(x, np.int8)
    dw = np.empty((CO, 3, 3, C), np.int64)
    _c().or_conv3x3_dw(_ptr(g64), _ptr(x8), _ptr(dw), N, H, W, C, CO)
    return dw


def linear_fwd(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """IntLinear (section 3.2.1): z[n][m] = sum_k x[n][k] W[m][k]. x int8 [N][K], w [M][K]."""
    N, K = x.shape
    M = w.shape[0]
    assert w.shape == (M, K)
    x8 = _as(x, np.int8)
    w32 = _as(w, np.int32)
    z = np.empty((N, M), np.int64)
    _c().or_linear_fwd(_ptr(x8), _ptr(w32), _ptr(z), N, K, M)
    return z


def linear_dx(e: np.ndarray, w: np.ndarray) -> np.ndarray:
    """e [N][M] times W [M][K] -> [N][K] int64 (the delta^fw product of section 3.3.4)."""
    N, M = e.shape
    K = w.shape[1]
    assert w.shape == (M, K)
    e64 = _as(e, np.int64)
    w32 = _as(w, np.int32)
    dx = np.empty((N, K), np.int64)
    _c().or_linear_dx(_ptr(e64), _ptr(w32), _ptr(dx), N, K, M)
    return dx


def linear_dw(e: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Weight gradient of IntLinear summed over the batch: dW[m][k] = sum_n e[n][m] x[n][k]."""
    N, M = e.shape
    K = x.shape[1]
    assert x.shape == (N, K)
    e64 = _as(e, np.int64)
    x8 = _as(x, np.int8)
    dw = np.empty((M, K), np.int64)
    _c().or_linear_dw(_ptr(e64), _ptr(x8), _ptr(dw), N, K, M)
    return dw


# ---------------------------------------------------------------------------------------------
# scalars and elementwise steps
# ---------------------------------------------------------------------------------------------

def idiv(a, b, mode: int = FLOOR):
    """Integer division by a positive divisor: floor (the paper's macro) or toward zero."""
    a = np.asarray(a, dtype=np.int64)
    b = np.asarray(b, dtype=np.int64)
    if np.any(b <= 0):
        raise ValueError("divisor must be positive")
    if mode == FLOOR:
        return a // b                      # numpy floor division: rounds toward minus infinity
    if mode == TRUNC:
        return np.sign(a) * (np.abs(a) // b)
    raise ValueError("unknown rounding mode")


def check_int32(a: np.ndarray, what: str) -> np.ndarray:
    a = np.asarray(a)
    if a.size and (a.min() < INT32_MIN or a.max() > INT32_MAX):
        raise OverflowError("%s does not fit int32 (range %d..%d)" % (what, a.min(), a.max()))
    return a


def scaling_factor_linear(m_prev: int) -> int:
    """SF = 2^8 * M_{l-1} for linear layers (section 3.2.1)."""
    return (1 << 8) * m_prev


def scaling_factor_conv(k: int, c_prev: int) -> int:
    """SF = 2^8 * K^2 * C_{l-1} for convolutional layers (section 3.2.1)."""
    return (1 << 8) * k * k * c_prev


def nitro_scaling(z, sf: int, mode: int = FLOOR):
    """NITRO-Scaling, Eq. 1: z* = z / SF rounded by the division rule."""
    return idiv(z, sf, mode)


def relu_mu(alpha_inv: int, mode: int = FLOOR) -> int:
    """Mean of NITRO-ReLU (section 3.2.2): the average of the four segment means
    {-127/alpha_inv, -127/(2 alpha_inv), 63, 127}, every division by the rounding rule."""
    segs = [int(idiv(-127, alpha_inv, mode)), int(idiv(-127, 2 * alpha_inv, mode)), 63, 127]
    return int(idiv(sum(segs), 4, mode))


def nitro_relu(zs, alpha_inv: int, mode: int = FLOOR):
    """NITRO-ReLU (section 3.2.2): max(x,-127)/alpha_inv - mu for x < 0, min(x,127) - mu for x >= 0."""
    zs = np.asarray(zs, dtype=np.int64)
    mu = relu_mu(alpha_inv, mode)
    neg = idiv(np.maximum(zs, -127), alpha_inv, mode) - mu
    pos = np.minimum(zs, 127) - mu
    return np.where(zs < 0, neg, pos)


def nitro_relu_grad(delta, zs, alpha_inv: int, mode: int = FLOOR, ste: bool = False):
    """Backward of NITRO-ReLU at the stored z* (the reading stated in the module docstring).
    ``ste=True`` is the alternative reading: a plain straight-through pass (gradient unchanged)
    on the leaky segment as well; the saturated segments still pass nothing."""
    delta = np.asarray(delta, dtype=np.int64)
    zs = np.asarray(zs, dtype=np.int64)
    slope = delta if ste else idiv(delta, alpha_inv, mode)
    out = np.where((zs >= 0) & (zs <= 127), delta, 0)
    out = np.where((zs < 0) & (zs >= -127), slope, out)
    return out


def maxpool2(a):
    """2x2 max-pool, stride 2 (Tab. 1 caption) on NHWC. Returns (pooled, window index 0..3 of the
    first maximum in row-major window order)."""
    a = np.asarray(a)
    N, H, W, C = a.shape
    v = a.reshape(N, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 2, 4, 5).reshape(N, H // 2, W // 2, 4, C)
    idx = np.argmax(v, axis=3)                # numpy returns the first occurrence of the maximum
    pooled = np.take_along_axis(v, idx[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return pooled, idx


def maxpool2_bwd(dp, idx, full_shape):
    """Route each pooled gradient to the window position that won the forward max."""
    N, H, W, C = full_shape
    dp = np.asarray(dp, dtype=np.int64)
    v = np.zeros((N, H // 2, W // 2, 4, C), np.int64)
    np.put_along_axis(v, idx[:, :, :, None, :], dp[:, :, :, None, :], axis=3)
    return v.reshape(N, H // 2, W // 2, 2, 2, C).transpose(0, 1, 3, 2, 4, 5).reshape(N, H, W, C)


def learning_pool_window(c: int, h: int, w: int, d_lr: int):
    """Window (kh, kw) of the learning layers' max-pool (the pooling of section 3.3 that turns a
    block's activations a_l into z^mp, d^lr of Tab. 6). Reading: starting from the whole
    resolution, the height and the width are halved in turn, the height first, until
    c * (h / kh) * (w / kw) <= d_lr or neither can be halved; d_lr = 0 means no pooling."""
    kh = kw = 1
    turn_h = True
    while d_lr > 0 and c * (h // kh) * (w // kw) > d_lr:
        can_h = (h // kh) % 2 == 0
        can_w = (w // kw) % 2 == 0
        if not (can_h or can_w):
            break
        if (turn_h and can_h) or not can_w:
            kh *= 2
        else:
            kw *= 2
        turn_h = not turn_h
    return kh, kw


def maxpool_window(a, kh: int, kw: int):
    """Non-overlapping kh x kw max-pool on NHWC. Returns (pooled, index 0 .. kh*kw-1 of the first
    maximum in row-major window order)."""
    a = np.asarray(a)
    N, H, W, C = a.shape
    v = a.reshape(N, H // kh, kh, W // kw, kw, C).transpose(0, 1, 3, 2, 4, 5)
    v = v.reshape(N, H // kh, W // kw, kh * kw, C)
    idx = np.argmax(v, axis=3)                # first occurrence of the maximum
    pooled = np.take_along_axis(v, idx[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return pooled, idx


def maxpool_window_bwd(dp, idx, full_shape, kh: int, kw: int):
    """Route each pooled gradient to the window position that won the forward max."""
    N, H, W, C = full_shape
    dp = np.asarray(dp, dtype=np.int64)
    v = np.zeros((N, H // kh, W // kw, kh * kw, C), np.int64)
    np.put_along_axis(v, idx[:, :, :, None, :], dp[:, :, :, None, :], axis=3)
    v = v.reshape(N, H // kh, W // kw, kh, kw, C).transpose(0, 1, 3, 2, 4, 5)
    return v.reshape(N, H, W, C)


def one_hot32(labels, G: int):
    """The custom one-hot target: 32 at the label, 0 elsewhere (section 3.3.4, Appendix A)."""
    labels = np.asarray(labels, dtype=np.int64)
    if labels.size and (labels.min() < 0 or labels.max() >= G):
        raise ValueError("label outside [0, G)")
    y = np.zeros((labels.shape[0], G), np.int64)
    y[np.arange(labels.shape[0]), labels] = 32
    return y


def loss_grad(yhat, labels, G: int):
    """Gradient of the RSS loss, Eq. 4, per sample: yhat - y."""
    return np.asarray(yhat, dtype=np.int64) - one_hot32(labels, G)


def predict(yhat) -> np.ndarray:
    """Predicted class per sample: the index of the largest prediction, the first one on ties."""
    return np.argmax(np.asarray(yhat), axis=1).astype(np.int32)


def amplification_factor(G: int) -> int:
    """NITRO Amplification Factor, Eq. 6: AF = 2^6 * G."""
    return (1 << 6) * G


def integer_sgd(w, dw, gamma_inv: int, lambda_inv: int, mode: int = FLOOR, eta_inv: int = -1):
    """IntegerSGD with weight decay (Alg. 1) in closed form:
    W' = W - (dW / gamma_inv + [eta_inv != 0] * W / eta_inv), with eta_inv = gamma_inv * lambda_inv
    unless an explicit eta_inv is given, every division by the rounding rule."""
    if gamma_inv < 1 or lambda_inv < 0:
        raise ValueError("gamma_inv >= 1 and lambda_inv >= 0 required")
    eta = gamma_inv * lambda_inv if eta_inv < 0 else eta_inv
    w = np.asarray(w, dtype=np.int64)
    decay = idiv(w, eta, mode) if eta != 0 else np.zeros_like(w)
    return check_int32(w - (idiv(dw, gamma_inv, mode) + decay), "updated weights")


def dropout_threshold(p_ppm: int) -> int:
    """The dropout probability p, given in parts per million, as a threshold on a 32-bit random
    number: floor(p_ppm 2^32 / 10^6)."""
    if not 0 <= p_ppm <= 1000000:
        raise ValueError("dropout rate outside [0, 10^6] ppm")
    return (p_ppm << 32) // 1000000


def dropout_keep(count: int, seed: int, step: int, block: int, p_ppm: int) -> np.ndarray:
    """Dropout mask of a block output with `count` elements (flat NHWC / [n][d] order), drawn
    with the counter-based generator Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): element i
    takes 64-bit word i mod 4 of the generator's output for counter (i div 4 + 1, block, step, 0)
    and key (seed, 0), and is kept when the word's upper 32 bits are at least the threshold.
    numpy's Philox bit generator (which steps its counter before each output) supplies the words."""
    if p_ppm == 0:
        return np.ones(count, bool)
    g = np.random.Philox(key=np.array([seed, 0], np.uint64),
                         counter=np.array([0, block, step, 0], np.uint64))
    words = g.random_raw((count + 3) // 4 * 4)[:count]
    return (words >> np.uint64(32)) >= np.uint64(dropout_threshold(p_ppm))


def kaiming_bound(fan_in: int) -> int:
    """Integer Kaiming bound (section 3.3.1): floor(128 * 1732 / (isqrt(fan_in) * 1000))."""
    return (128 * 1732) // (math.isqrt(fan_in) * 1000)


# ---------------------------------------------------------------------------------------------
# integer pre-processing of the input data (Appendix A)
# ---------------------------------------------------------------------------------------------

@dataclass
class Preprocessed:
    mu: int                   # integer mean of the dataset
    omega: int                # integer mean absolute deviation (the divisor used: at least 1)
    xhat: np.ndarray          # normalised data, int8
    saturated: int            # elements whose normalised value left [-127, 127]


def preprocess(x, mode: int = FLOOR) -> Preprocessed:
    """Appendix A: mu = sum_i x_i / N, omega = sum_i |x_i - mu| / N, xhat_i = (x_i - mu) 51 / omega,
    every division by the rounding rule, over all N elements of the dataset.
    Readings: mu and omega are single numbers for the whole dataset; a dataset whose omega
    rounds to 0 is divided by 1; xhat is stored as int8, so values outside [-127, 127] are
    clamped to it (and counted)."""
    x = np.asarray(x, dtype=np.int64).reshape(-1)
    n = x.size
    if n == 0:
        raise ValueError("empty dataset")
    mu = int(idiv(x.sum(), n, mode))
    omega = int(idiv(np.abs(x - mu).sum(), n, mode))
    div = max(omega, 1)
    v = idiv((x - mu) * 51, div, mode)
    sat = int(np.count_nonzero((v < -127) | (v > 127)))
    return Preprocessed(mu=mu, omega=div, xhat=np.clip(v, -127, 127).astype(np.int8), saturated=sat)


# ---------------------------------------------------------------------------------------------
# whole-step composition (section 3.3, training procedure)
# ---------------------------------------------------------------------------------------------

@dataclass
class LayerRecord:
    x: np.ndarray             # layer input (int8 values)
    z: np.ndarray             # pre-activation, int64
    zs: np.ndarray            # rescaled pre-activation z*
    a: np.ndarray             # NITRO-ReLU output (int8 values)


@dataclass
class BlockRecord:
    layers: List[LayerRecord] = field(default_factory=list)
    out: Optional[np.ndarray] = None        # block output (pooled if the block pools), int8
    pool_idx: Optional[np.ndarray] = None
    keep: Optional[np.ndarray] = None       # dropout mask of the block output (None: no dropout)
    yhat: Optional[np.ndarray] = None       # learning-layer prediction, int32 values
    e: Optional[np.ndarray] = None          # local loss gradient
    dw_lr: Optional[np.ndarray] = None
    f: Optional[np.ndarray] = None          # learning-layer input: the block output, max-pooled
    #                                         to at most d_lr features when d_lr is set
    f_idx: Optional[np.ndarray] = None      # its window argmax (None: f is the block output)
    f_window: tuple = (1, 1)
    delta_fw: Optional[np.ndarray] = None   # gradient at the learning layer's input f
    g: List[np.ndarray] = field(default_factory=list)     # gradient at each layer's z (after ReLU')
    dw: List[np.ndarray] = field(default_factory=list)    # per forward layer, int64
    dx: Optional[np.ndarray] = None         # input gradient of the first layer (when asked for)


def _is_conv(w: np.ndarray) -> bool:
    return w.ndim == 4


def layer_forward(x, w, alpha_inv: int, mode: int) -> LayerRecord:
    """One forward layer: IntConv2D / IntLinear -> NITRO-Scaling -> NITRO-ReLU."""
    if _is_conv(w):
        z = conv3x3_fwd(x, w)
        sf = scaling_factor_conv(3, w.shape[3])
    else:
        z = linear_fwd(x, w)
        sf = scaling_factor_linear(w.shape[1])
    zs = nitro_scaling(z, sf, mode)
    a = nitro_relu(zs, alpha_inv, mode)
    assert a.min() >= -128 and a.max() <= 127
    return LayerRecord(x=np.asarray(x), z=z, zs=zs, a=a.astype(np.int8))


def block_forward(x, ws: list, maxpool: bool, alpha_inv: int, mode: int) -> BlockRecord:
    rec = BlockRecord()
    cur = x
    for w in ws:
        lr = layer_forward(cur, w, alpha_inv, mode)
        rec.layers.append(lr)
        cur = lr.a
    if maxpool:
        cur, rec.pool_idx = maxpool2(cur)
    rec.out = np.asarray(cur, dtype=np.int8)
    return rec


def learning_forward(f, w_lr, mode: int):
    """Learning / output layer: IntLinear(d -> G) followed by NITRO-Scaling with SF = 2^8 d."""
    z = linear_fwd(f, w_lr)
    return check_int32(nitro_scaling(z, scaling_factor_linear(w_lr.shape[1]), mode), "yhat")


def block_backward(rec: BlockRecord, ws: list, delta_out, maxpool: bool, alpha_inv: int,
                   mode: int, want_dx: bool = False, ste: bool = False) -> None:
    """Back-propagate the gradient at the block output through the forward layers of the block,
    using the weights from before the update. Fills rec.g, rec.dw (and rec.dx). ``ste`` selects
    the straight-through reading of the NITRO-ReLU backward (nitro_relu_grad)."""
    J = len(ws)
    last = rec.layers[-1]
    d = np.asarray(delta_out, dtype=np.int64)
    if maxpool:
        d = maxpool2_bwd(d, rec.pool_idx, last.a.shape)
    d = d.reshape(last.zs.shape)
    gs = [None] * J
    dws = [None] * J
    g = check_int32(nitro_relu_grad(d, last.zs, alpha_inv, mode, ste), "ReLU gradient")
    for j in range(J - 1, -1, -1):
        gs[j] = g
        ly = rec.layers[j]
        if _is_conv(ws[j]):
            dws[j] = conv3x3_dw(g, ly.x)
        else:
            dws[j] = linear_dw(g, ly.x)
        if j > 0 or want_dx:
            if _is_conv(ws[j]):
                dx = conv3x3_dx(g, ws[j])
            else:
                dx = linear_dx(g, ws[j])
            if j > 0:
                dx = check_int32(dx, "input gradient")
                g = check_int32(nitro_relu_grad(dx, rec.layers[j - 1].zs, alpha_inv, mode, ste),
                                "ReLU gradient")
            else:
                rec.dx = dx       # leaves the block: never used by the method, kept in int64
    rec.g = gs
    rec.dw = dws


@dataclass
class Hyper:
    gamma_inv: int
    lambda_inv_fw: int
    lambda_inv_lr: int
    alpha_inv: int
    n_classes: int
    mode: int = FLOOR
    af_classes: int = 0          # G for the amplification factor when n_classes == 0
    eta_fw: int = -1             # explicit eta overrides (< 0: gamma * lambda)
    eta_lr: int = -1
    d_lr: int = 0                # learning-layer input size of conv blocks (0: the block output)
    dropout_conv_ppm: int = 0    # dropout rate p_c of conv blocks' outputs (parts per million)
    dropout_lin_ppm: int = 0     # dropout rate p_l of linear blocks' outputs
    dropout_seed: int = 0        # key of the dropout generator
    dropout_step: int = 0        # counter of the first training iteration
    # alternative readings (both off by default):
    relu_grad_ste: bool = False  # NITRO-ReLU backward passes the gradient unchanged on its leaky
    #                              segment (straight through) instead of dividing by alpha_inv
    delta_fw_post_update: bool = False   # delta^fw from the learning weights after their update
    #                              (the literal order of the training procedure in section 3.3)

    @property
    def gamma_fw(self) -> int:
        """gamma_inv^fw = AF * gamma_inv^lr (section 3.3.4, Eq. 6)."""
        return amplification_factor(self.n_classes or self.af_classes) * self.gamma_inv


@dataclass
class StepRecord:
    blocks: List[BlockRecord]
    head_yhat: Optional[np.ndarray] = None
    head_e: Optional[np.ndarray] = None
    head_dw: Optional[np.ndarray] = None


class OracleNet:
    """The network state and one training iteration exactly as section 3.3 describes it.

    ``weights`` follows the draw order of the workload module: per block its forward layers, then
    its learning layer (if any); then the output head (if any)."""

    def __init__(self, block_specs, head: bool, weights: list, hp: Hyper):
        # block_specs: list of (n_forward_layers, maxpool, has_learning)
        self.specs = list(block_specs)
        self.head = head
        self.hp = hp
        self.w = [np.asarray(w, dtype=np.int32).copy() for w in weights]
        self.index = []       # per block: (list of forward-layer weight indices, learning index or None)
        i = 0
        for nl, _, has_lr in self.specs:
            fw = list(range(i, i + nl))
            i += nl
            lr = None
            if has_lr:
                lr = i
                i += 1
            self.index.append((fw, lr))
        self.head_index = i if head else None
        assert len(self.w) == i + (1 if head else 0)
        self.steps = 0                # training iterations done (the dropout counter)

    def forward(self, x, train: bool = False) -> List[BlockRecord]:
        """The forward layers of every block; in training, a block's output then takes dropout
        (rate p_c for conv blocks, p_l for linear blocks; dropped elements become 0 for the next
        block and the learning layer alike, and pass no gradient back)."""
        recs = []
        cur = x
        hp = self.hp
        for b, (nl, pool, _) in enumerate(self.specs):
            fw, _ = self.index[b]
            ws = [self.w[k] for k in fw]
            if not _is_conv(ws[0]) and cur.ndim == 4:
                cur = cur.reshape(cur.shape[0], -1)       # flatten in (h, w, c) order
            rec = block_forward(cur, ws, pool, hp.alpha_inv, hp.mode)
            p = hp.dropout_conv_ppm if _is_conv(ws[0]) else hp.dropout_lin_ppm
            if train and p > 0:
                keep = dropout_keep(rec.out.size, hp.dropout_seed, hp.dropout_step + self.steps,
                                    b, p).reshape(rec.out.shape)
                rec.keep = keep
                rec.out = np.where(keep, rec.out, 0).astype(np.int8)
            recs.append(rec)
            cur = rec.out
        return recs

    def train_step(self, x, labels) -> StepRecord:
        hp = self.hp
        mode = hp.mode
        G = hp.n_classes
        # forward pass through every block's forward layers (section 3.3, first paragraph)
        recs = self.forward(x, train=True)
        step = StepRecord(blocks=recs)
        new_w = [w.copy() for w in self.w]
        # output layers: global gradient, weight gradient, IntegerSGD with gamma^lr
        if self.head:
            h = self.head_index
            f = recs[-1].out.reshape(recs[-1].out.shape[0], -1)
            step.head_yhat = learning_forward(f, self.w[h], mode)
            step.head_e = check_int32(loss_grad(step.head_yhat, labels, G), "loss gradient")
            step.head_dw = linear_dw(step.head_e, f)
            new_w[h] = integer_sgd(self.w[h], step.head_dw, hp.gamma_inv, hp.lambda_inv_lr, mode,
                                   hp.eta_lr).astype(np.int32)
        # local training of every block (independent of the others)
        for b, (nl, pool, has_lr) in enumerate(self.specs):
            rec = recs[b]
            fw, lr = self.index[b]
            if not has_lr:
                continue
            rec.f = rec.out
            if rec.out.ndim == 4 and hp.d_lr > 0:
                N_, H_, W_, C_ = rec.out.shape
                rec.f_window = learning_pool_window(C_, H_, W_, hp.d_lr)
                if rec.f_window != (1, 1):
                    rec.f, rec.f_idx = maxpool_window(rec.out, *rec.f_window)
            f = rec.f.reshape(rec.f.shape[0], -1)
            w_lr = self.w[lr]
            rec.yhat = learning_forward(f, w_lr, mode)
            rec.e = check_int32(loss_grad(rec.yhat, labels, G), "loss gradient")
            rec.dw_lr = linear_dw(rec.e, f)
            new_w[lr] = integer_sgd(w_lr, rec.dw_lr, hp.gamma_inv, hp.lambda_inv_lr, mode,
                                    hp.eta_lr).astype(np.int32)
            w_delta = new_w[lr] if hp.delta_fw_post_update else w_lr       # default: pre-update
            rec.delta_fw = check_int32(linear_dx(rec.e, w_delta), "delta_fw")
            d_out = rec.delta_fw.reshape(rec.f.shape)
            if rec.f_idx is not None:              # back through the learning layers' pooling
                d_out = maxpool_window_bwd(d_out, rec.f_idx, rec.out.shape, *rec.f_window)
            if rec.keep is not None:               # dropped outputs pass no gradient
                d_out = np.where(rec.keep, d_out, 0)
            block_backward(rec, [self.w[k] for k in fw], d_out,
                           pool, hp.alpha_inv, mode, ste=hp.relu_grad_ste)
            for j, k in enumerate(fw):
                new_w[k] = integer_sgd(self.w[k], rec.dw[j], hp.gamma_fw, hp.lambda_inv_fw, mode,
                                       hp.eta_fw).astype(np.int32)
        self.w = new_w
        self.steps += 1
        return step

    def infer(self, x):
        """Inference: the forward pass, then the network's prediction yhat (the output layer's,
        or without one the last block's learning layer's) and the predicted class, the first
        maximum of each row (argmax). Returns (yhat, pred)."""
        recs = self.forward(x)
        last = recs[-1]
        if self.head:
            f = last.out.reshape(last.out.shape[0], -1)
            w = self.w[self.head_index]
        else:
            f = last.out
            if f.ndim == 4 and self.hp.d_lr > 0:
                N_, H_, W_, C_ = f.shape
                win = learning_pool_window(C_, H_, W_, self.hp.d_lr)
                if win != (1, 1):
                    f, _ = maxpool_window(f, *win)
            f = f.reshape(f.shape[0], -1)
            w = self.w[self.index[-1][1]]
        yhat = learning_forward(f, w, self.hp.mode)
        return yhat, predict(yhat)

    def stress_repeat(self, x, delta) -> BlockRecord:
        """The single-layer stress case: forward, then back-propagate a given gradient at the
        NITRO-ReLU output (input gradient included), then IntegerSGD with gamma^fw."""
        hp = self.hp
        fw, _ = self.index[0]
        ws = [self.w[k] for k in fw]
        rec = block_forward(x, ws, self.specs[0][1], hp.alpha_inv, hp.mode)
        block_backward(rec, ws, delta, self.specs[0][1], hp.alpha_inv, hp.mode, want_dx=True,
                       ste=hp.relu_grad_ste)
        for j, k in enumerate(fw):
            self.w[k] = integer_sgd(self.w[k], rec.dw[j], hp.gamma_fw, hp.lambda_inv_fw, hp.mode,
                                    hp.eta_fw).astype(np.int32)
        return rec


# ---------------------------------------------------------------------------------------------
# single-output evaluations, for checks at full size on sampled positions
# ---------------------------------------------------------------------------------------------

def conv3x3_fwd_at(x, w, n, h, wq, co) -> int:
    N, H, W, C = x.shape
    acc = 0
    for r in range(3):
        for s in range(3):
            hh, ww = h + r - 1, wq + s - 1
            if 0 <= hh < H and 0 <= ww < W:
                acc += int(np.dot(x[n, hh, ww, :].astype(np.int64), w[co, r, s, :].astype(np.int64)))
    return acc


def conv3x3_dx_at(g, w, n, h, wq, ci) -> int:
    N, H, W, CO = g.shape
    acc = 0
    for r in range(3):
        for s in range(3):
            ho, wo = h - r + 1, wq - s + 1
            if 0 <= ho < H and 0 <= wo < W:
                acc += int(np.dot(g[n, ho, wo, :].astype(np.int64), w[:, r, s, ci].astype(np.int64)))
    return acc


def conv3x3_dw_at(g, x, co, r, s, ci) -> int:
    N, H, W, C = x.shape
    gp = np.zeros((N, H + 2, W + 2), np.int64)
    gp[:, 1:H + 1, 1:W + 1] = g[:, :, :, co]
    # dW[co][r][s][ci] = sum_{n,h,w} g[n,h,w,co] x[n,h+r-1,w+s-1,ci]
    #                 = sum_{n,h',w'} g[n,h'-r+1,w'-s+1,co] x[n,h',w',ci]
    gs = gp[:, 2 - r:2 - r + H, 2 - s:2 - s + W]
    return int(np.sum(gs * x[:, :, :, ci].astype(np.int64)))
