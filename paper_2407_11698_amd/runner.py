"""Drive the C ABI for a whole workload: build the block / network descriptors from a workload
description, hold weights and the workspace in torch device memory, and call nitro_train_step
(or the block-level calls for the single-layer stress case). Marshalling only."""
from __future__ import annotations

from typing import List

import numpy as np
import torch

from . import nitro as N
from .workloads import Conv3x3, Workload


# weight initialisation bound (section 3.3.1), computed by the library
kaiming_bound = N.kaiming_bound


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
                                  wl.n_classes if blk.learning else 0, wl.alpha_inv, round_mode,
                                  wl.d_lr))
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
        # every weight a view of one flat int32 buffer (each at a multiple of 64 elements), so that
        # a caller can save or restore all of them with one copy
        sizes = [int(np.prod(np.shape(w))) for w in weights]
        offs, o = [], 0
        for n in sizes:
            offs.append(o)
            o += (n + 63) // 64 * 64
        self.w_flat = torch.zeros(o, dtype=torch.int32, device=self.dev)
        self.w = []
        for w, off, n in zip(weights, offs, sizes):
            t = self.w_flat[off:off + n].view(np.shape(w))
            t.copy_(_dev(np.asarray(w, dtype=np.int32), self.dev))
            self.w.append(t)
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
        self.hp = N.hparams(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr,
                            dropout_conv_ppm=wl.dropout_conv_ppm, dropout_lin_ppm=wl.dropout_lin_ppm,
                            dropout_seed=wl.dropout_seed)
        self.steps = 0                 # iterations taken: the dropout generator's step counter

    def step(self, x: torch.Tensor, y: torch.Tensor) -> None:
        self.hp.dropout_step = self.steps
        self.ctx.train_step(self.nd, self.params, self.workspace, x, y, self.hp)
        self.steps += 1

    def step_graph(self, x: torch.Tensor, y: torch.Tensor) -> None:
        """One iteration replayed from the context's captured graph for these buffers (captured
        on the first call with them; up to 16 buffer sets keep graphs of their own). The dropout
        step counter is part of a graph's arguments, so workloads with dropout take the eager
        path instead."""
        if self.wl.dropout_conv_ppm or self.wl.dropout_lin_ppm:
            return self.step(x, y)
        self.ctx.train_step_graph(self.nd, self.params, self.workspace, x, y, self.hp)
        self.steps += 1

    def prepare_graph(self, x: torch.Tensor, y: torch.Tensor) -> None:
        """Capture (without running) the graph step_graph replays for these buffers."""
        if self.wl.dropout_conv_ppm or self.wl.dropout_lin_ppm:
            return
        self.ctx.train_step_graph_prepare(self.nd, self.params, self.workspace, x, y, self.hp)

    def infer(self, x: torch.Tensor):
        """Inference with the current weights: (yhat [n][G] int32, predicted class [n] int32)."""
        yhat = torch.empty((self.wl.batch, self.wl.n_classes), dtype=torch.int32, device=self.dev)
        pred = torch.empty((self.wl.batch,), dtype=torch.int32, device=self.dev)
        self.ctx.net_infer(self.nd, self.params, self.workspace, x, yhat, pred)
        return yhat, pred

    def view(self, b: int) -> dict:
        """Block b's tensors from the last step, as torch views of the workspace: "a_out",
        "act" (list, None for the last layer), "code" (list), "yhat", "e", "dw" (list), "dw_lr"."""
        ptrs = N.net_block_view(self.nd, self.workspace, b)
        blk = self.wl.blocks[b]
        (inp, out) = self.wl.block_shapes()[b]
        n, G = self.wl.batch, self.wl.n_classes
        conv = isinstance(blk.layers[0], Conv3x3)
        full = []                    # per layer: output shape at full resolution
        for ly in blk.layers:
            full.append((n, inp[1], inp[2], ly.c_out) if conv else (n, ly.d_out))
        a_shape = (n, out[1], out[2], out[0]) if conv else (n,) + tuple(out)
        last = len(blk.layers) - 1
        res = {"a_out": self._at(ptrs["a_out"], a_shape, torch.int8),
               "act": [self._at(ptrs["act"][j], full[j], torch.int8) if j < last else None
                       for j in range(len(blk.layers))],
               "code": [self._at(ptrs["code"][j], a_shape if (j == last and blk.maxpool) else full[j],
                                 torch.uint8) for j in range(len(blk.layers))],
               "yhat": self._at(ptrs["yhat"], (n, G), torch.int32),
               "e": self._at(ptrs["e"], (n, G), torch.int32),
               "dw": [self._at(ptrs["dw"][j], tuple(w.shape), torch.int64)
                      for j, w in enumerate(self.w[self._first_weight(b):self._first_weight(b) + len(blk.layers)])],
               "dw_lr": self._at(ptrs["dw_lr"], (G, self.wl.learning_dim(b)), torch.int64)}
        return res

    def head_view(self) -> dict:
        ptrs = N.net_head_view(self.nd, self.workspace)
        n, G, d = self.wl.batch, self.wl.n_classes, self.wl.head_dim()
        return {"yhat": self._at(ptrs["yhat"], (n, G), torch.int32),
                "e": self._at(ptrs["e"], (n, G), torch.int32),
                "dw": self._at(ptrs["dw"], (G, d), torch.int64)}

    def _first_weight(self, b: int) -> int:
        k = 0
        for blk in self.wl.blocks[:b]:
            k += len(blk.layers) + (1 if blk.learning else 0)
        return k

    def _at(self, ptr: int, shape, dtype) -> torch.Tensor:
        off = ptr - self.workspace.data_ptr()
        nb = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        return self.workspace[off:off + nb].view(dtype).view(shape)

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
        self.hp = N.hparams(wl.gamma_inv, wl.lambda_inv_fw, wl.lambda_inv_lr,
                            af_classes=wl.af_classes)

    def repeat(self, x: torch.Tensor, delta: torch.Tensor, want_dx: bool = True,
               taps: dict = None) -> None:
        """Forward, back-propagation of `delta` (the int64 input gradient when want_dx), then
        IntegerSGD with the forward layers' amplified rate. `taps` adds extra outputs (the
        gradient at the pre-activation: {"g": [tensor]})."""
        t = dict(taps or {})
        if want_dx:
            t["dx"] = self.dx
        self.ctx.block_forward(self.desc, [self.w], x, self.a, self.state)
        self.ctx.block_backward(self.desc, [self.w], None, x, self.a, None, delta, self.state,
                                [self.dw], None, t or None)
        self.ctx.block_sgd_step(self.desc, [self.w], None, [self.dw], None, self.hp)
