"""Where the two readings of the paper's integer division diverge, end to end.

The paper defines its division as the floor (its macro, used in every formula), while its text on
IntegerSGD speaks of truncation (weights below eta_inv get no decay; too large a gamma_inv
"truncates" updates to zero). The library runs either rounding for every division of the step.
This study trains each workload twice on the GPU, from the same initial weights on the same
seeded batches, once per rounding mode, and reports per step:
  * out_diff      fraction of the last block's output elements that differ between the modes;
  * w_diff        fraction of all weights that differ;
  * w_absdiff     mean |W_floor - W_trunc| over all weights;
  * unchanged     per mode, the fraction of weights the step left unchanged (truncation rounds
                  small updates and small decays to zero; the floor rounds negative ones to -1);
  * pred_agree    agreement of the two networks' predicted classes on a held-out batch.

Usage (one GPU): python -m paper_2407_11698_amd.study_rounding [--steps 10]; prints one JSON line
per workload.
"""
from __future__ import annotations

import argparse
import json

import numpy as np
import torch

from . import nitro as N
from . import runner
from . import workloads as WL


def study(wl, steps: int) -> dict:
    dev = torch.device("cuda", 0)
    dr = WL.draw_workload(wl, runner.kaiming_bound, steps=steps + 1)
    xt = torch.from_numpy(dr.batches[-1][0]).to(dev)
    nets = {m: runner.GpuNet(wl, dr.weights, rm) for m, rm in (("floor", N.ROUND_FLOOR),
                                                                 ("trunc", N.ROUND_TRUNC))}
    last = len(wl.blocks) - 1
    rows = []
    for s in range(steps):
        x, y = (torch.from_numpy(a).to(dev) for a in dr.batches[s])
        before = {m: [w.clone() for w in n.w] for m, n in nets.items()}
        for n in nets.values():
            n.step(x, y)
            n.ctx.sync()
        out = {m: n.block_output(last).clone() for m, n in nets.items()}
        wf = torch.cat([w.reshape(-1).to(torch.int64) for w in nets["floor"].w])
        wt = torch.cat([w.reshape(-1).to(torch.int64) for w in nets["trunc"].w])
        unchanged = {}
        for m, n in nets.items():
            same = sum(int((a == b).sum().item()) for a, b in zip(n.w, before[m]))
            unchanged[m] = round(same / wf.numel(), 5)
        preds = {}
        for m, n in nets.items():
            _, p = n.infer(xt)
            n.ctx.sync()
            preds[m] = p.cpu().numpy()
        rows.append({"step": s,
                     "out_diff": round(float((out["floor"] != out["trunc"]).float().mean()), 5),
                     "w_diff": round(float((wf != wt).float().mean()), 5),
                     "w_absdiff": round(float((wf - wt).abs().float().mean()), 3),
                     "unchanged": unchanged,
                     "pred_agree": round(float(np.mean(preds["floor"] == preds["trunc"])), 4)})
    return {"workload": wl.name, "batch": wl.batch, "steps": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=10)
    args = ap.parse_args()
    for wl in (WL.TINY_CNN, WL.MLP, WL.SMALL_CNN, WL.VGG_CNN, WL.VGG8B, WL.MLP3):
        print(json.dumps(study(wl, args.steps)), flush=True)


if __name__ == "__main__":
    main()
