"""Drive the C ABI for a whole workload: build the block / network descriptors from a workload
description, hold weights and the workspace in torch device memory, and call nitro_train_step
(or the block-level calls for the single-layer stress case). Marshalling only."""
from __future__ import annotations

import math
from typing import List

import numpy as np
import torch

from . import nitro as N
from .workloads import Conv3x3, Workload


def kaiming_bound(fan_in: int) -> int:
    """Integer Kaiming bound of section 3.3.1: floor(128 * 1732 / (isqrt(fan_in) * 1000))."""
    return (128 * 1732) // (math.isqrt(fan_in) * 1000)


def block_descs(wl: Workload, round_mode: int = N.ROUND_FLOOR) -> List[N.BlockDesc]:
    descs = []
    for (inp, _), blk in zip(wl.block_shapes(), wl.blocks):
        if isinstance(blk.layers[0], Conv3x3):
            _, h, w = inp
            layers = [N.layer(N.CONV3X3, ly.c_in, ly.c_out) for ly in blk.layers]
        else:
            h = w = 1
            layers = [N.layer(N.LINEAR, ly.d_in, ly.d_out) for ly in blk.layers]
        descs.append(N.block_desc(wl.batch, h, w, layers, blk.maxpool,
                                  wl.n_classes if blk.learning else 0, wl.alpha_inv, round_mode))
    return descs


def _dev(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class GpuNet:
    """A network whose every block has a learning layer; weights in draw order (per block: the
    forward layers, then the learning layer; then the output head)."""

    def __init__(self, wl: Workload, weights: list, round_mode: int = N.ROUND_FLOOR,
                 device: int = 0, ctx: N.Context = None):
        self.wl = wl
        self.dev = torch.device("cuda", device)
        self.ctx = ctx or N.Context(device)
        self.descs = block_descs(wl, round_mode)
        self.nd = N.net_desc(self.descs, wl.head)
        self.w = [_dev(w, self.dev) for w in weights]
        self.params = N.NetParams()
        k = 0
        for b, blk in enumerate(wl.blocks):
            for j in range(len(blk.layers)):
                self.params.w[b][j] = self.w[k].data_ptr()
                k += 1
            self.params.w_lr[b] = self.w[k].data_ptr()
            k += 1
        if wl.head:
            self.params.w_head = self.w[k].data_ptr()
            k += 1
        assert k == len(self.w)
        self.workspace = torch.empty(N.net_query(self.nd), dtype=torch.uint8, device=self.dev)
        self.hp = N.HParams(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr, 0, -1, -1)

    def step(self, x: torch.Tensor, y: torch.Tensor) -> None:
        self.ctx.train_step(self.nd, self.params, self.workspace, x, y, self.hp)

    def step_graph(self, x: torch.Tensor, y: torch.Tensor) -> None:
        """One iteration replayed from the context's captured graph for these buffers (captured
        on the first call with them; up to 16 buffer sets keep graphs of their own)."""
        self.ctx.train_step_graph(self.nd, self.params, self.workspace, x, y, self.hp)

    def block_output(self, b: int) -> torch.Tensor:
        """Block b's output from the last step (int8, NHWC or [n][d])."""
        ptr = self.ctx.net_block_output_ptr(self.nd, self.workspace, b)
        off = ptr - self.workspace.data_ptr()
        _, out = self.wl.block_shapes()[b]
        shape = (self.wl.batch,) + ((out[1], out[2], out[0]) if len(out) == 3 else out)
        n = int(np.prod(shape))
        return self.workspace[off:off + n].view(torch.int8).view(shape)

    def weights_np(self) -> list:
        return [w.cpu().numpy() for w in self.w]


class GpuConvStress:
    """The single conv-layer stress case: forward, back-propagation of a given gradient at the
    NITRO-ReLU output (input gradient included), IntegerSGD with gamma^fw = AF * gamma."""

    def __init__(self, wl: Workload, weight: np.ndarray, round_mode: int = N.ROUND_FLOOR,
                 device: int = 0, ctx: N.Context = None):
        self.wl = wl
        self.dev = torch.device("cuda", device)
        self.ctx = ctx or N.Context(device)
        self.desc = block_descs(wl, round_mode)[0]
        self.round = round_mode
        ly = wl.blocks[0].layers[0]
        c, h, w = wl.in_shape
        self.w = _dev(weight, self.dev)
        self.state = torch.empty(N.block_query(self.desc), dtype=torch.uint8, device=self.dev)
        self.a = torch.empty((wl.batch, h, w, ly.c_out), dtype=torch.int8, device=self.dev)
        self.dw = torch.empty((ly.c_out, 3, 3, ly.c_in), dtype=torch.int64, device=self.dev)
        self.dx = torch.empty((wl.batch, h, w, ly.c_in), dtype=torch.int64, device=self.dev)
        self.gamma_fw = (1 << 6) * wl.af_classes * wl.gamma_inv

    def repeat(self, x: torch.Tensor, delta: torch.Tensor, want_dx: bool = True) -> None:
        self.ctx.block_forward(self.desc, [self.w], x, self.a, self.state)
        self.ctx.block_backward(self.desc, [self.w], None, x, self.a, None, delta, self.state,
                                [self.dw], None, {"dx": self.dx} if want_dx else None)
        self.ctx.integer_sgd_step(self.w, self.dw, self.gamma_fw, self.wl.lambda_inv_fw,
                                  round_mode=self.round)
