"""Benchmark: images/s of the NITRO-D integer training iteration on one MI355X.

Workload: the VGG-style integer CNN (3x32x32 int8 inputs, batch 256, four blocks of two 3x3
convolutions 3-64-64, 64-128-128, 128-256-256, 256-512-512, 2x2 max-pool and a learning layer to
100 classes per block), trained with nitro_train_step. Inputs are seeded synthetic data already
resident in HBM. The timed loop replays the ten-step trajectory the parity tests check: every ten
steps the weights are reset to their initial values, so each timed step is one of those ten
verified iterations.

Prints one JSON line with the throughput, the roofline position of the dominant kernel (its own
device time inside the timed region, from timestamps its workgroups record; beside it, the same
kernel's time per launch in a few iterations run afterwards with every block on one stream, and
its HBM bytes per launch from the hardware-counter summary under profiles/ while that kernel's
source is unchanged), the single conv-layer stress case's kernels measured alone after the timed
region, and the CPU oracle's throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_INT8_TOPS = 5000.0          # dense int8 MFMA, TOP/s
PEAK_HBM_GBS = 8000.0

# timed kernel classes of the library (nitro_kernel_time) and the HIP kernels they bracket
KERNEL_CLASSES = {0: "k_conv_tile<fwd>", 1: "k_conv_tile<dx>", 2: "k_conv_dw_planes"}


def conv_layer_ops(wl):
    """Algorithmic ops (2 x MACs, each GEMM counted once, no limb passes) per training iteration
    of the conv GEMMs that run on each timed MFMA kernel class.

    A layer with N*H*W output pixels, C_in inputs and C_out outputs has N*H*W*C_out*9*C_in MACs
    in each of its forward, input-gradient and weight-gradient GEMMs. The input gradient is
    computed for every layer but the first of a block (nothing leaves a block). The library
    routes a layer to the timed kernels when its shape fits them (forward and input gradient:
    128 % W == 0 and the GEMM's K channels 16, 32 or a multiple of 64, an input with fewer than
    16 channels being zero-padded to 16; weight gradient: C_out a multiple of 16 and W <= 62).
    Only the layer's own MACs are counted, not the padding."""
    from paper_2407_11698_amd.workloads import Conv3x3
    ops = {name: 0 for name in KERNEL_CLASSES.values()}
    for (inp, _), blk in zip(wl.block_shapes(), wl.blocks):
        if not isinstance(blk.layers[0], Conv3x3):
            continue
        _, h, w = inp
        for j, ly in enumerate(blk.layers):
            macs = wl.batch * h * w * ly.c_out * 9 * ly.c_in
            pool = blk.maxpool and j == len(blk.layers) - 1
            tiles = 128 % w == 0
            kok = lambda c: c in (16, 32) or c % 64 == 0
            if tiles and (kok(ly.c_in) or ly.c_in < 16) and ly.c_out % 16 == 0:
                ops["k_conv_tile<fwd>"] += 2 * macs
            if j > 0 and tiles and kok(ly.c_out) and ly.c_in % 16 == 0:
                ops["k_conv_tile<dx>"] += 2 * macs
            if ly.c_out % 16 == 0 and w <= 62:
                ops["k_conv_dw_planes"] += 2 * macs
    return ops


def recorded_traffic(kernel: str):
    """HBM bytes per launch of `kernel` in the training iteration, from the hardware-counter
    summary under profiles/ (FETCH_SIZE and WRITE_SIZE passes, each calibrated by a copy of
    known size); None when there is no summary or the kernel's source has changed since."""
    import hashlib
    tag = kernel.replace("<", "_").replace(">", "")
    path = os.path.join(ROOT, "profiles", "%s_vgg_cnn_b256_traffic.txt" % tag)
    try:
        kv = dict(line.split(": ", 1) for line in open(path).read().splitlines() if ": " in line)
        h = hashlib.sha256()
        for f in kv["sources"].split():
            h.update(open(os.path.join(ROOT, f), "rb").read())
    except (OSError, KeyError, ValueError):
        return None
    if kv.get("kernel") != kernel or h.hexdigest() != kv.get("sources_sha256"):
        return None
    return int(float(kv["traffic_bytes_per_launch"]))


def limbs_for(m: int) -> int:
    """Balanced signed base-256 int8 limbs needed for magnitudes up to m (|v| <= m)."""
    return 1 if m <= 127 else 2 if m <= 32639 else 3 if m <= 8355711 else 4


# The library's input and weight gradients of the single layer take g in two limbs plus an
# offset correction when 32639 < max|g| <= 32768 and at most this many entries of g equal 32768
# (three limbs otherwise).
G_OFFSET_CAP = 16384


def offset_g_limbs(g) -> int:
    """Limb passes over g of the single layer's input and weight gradients."""
    m = int(g.abs().max().item())
    if 32639 < m <= 32768 and int((g == 32768).sum().item()) <= G_OFFSET_CAP:
        return 2
    return limbs_for(m)


def stress_layer(reps: int):
    """The single conv-layer stress case (256x256x32x32 int8 activations, conv 256 -> 256, int32
    error signal in [-2^15, 2^15] at the NITRO-ReLU output), `reps` cumulative repeats, each a
    forward, the back-propagation of the error signal (weight and int64 input gradients) and the
    IntegerSGD step with the amplified rate, run alone on the GPU after the training iterations.

    Each repeat is timed whole with HIP events on the library's stream (every kernel of the
    repeat, IntegerSGD included), and its three conv GEMM kernels by their own device time; the
    repeat's g (limb passes) comes from an untimed replay of it from the same weights.
    Algorithmic ops count each GEMM once (2 x N*H*W*C_out*9*C_in, three GEMMs per repeat); MFMA
    ops count every limb pass the kernel executes, from the repeat's own max|W| and g (the input
    gradient's kernel time excludes the two small kernels of g's offset form, which the whole
    repeat includes; the weight gradient's, the split-K sums and their offset term). The
    weights leave int8 after the first repeat, so repeat 1 and the steady state (median over the
    later repeats) are reported separately."""
    import torch
    from paper_2407_11698_amd import runner
    from paper_2407_11698_amd import workloads as WL
    wl = WL.CONV_STRESS
    dr = WL.draw_workload(wl, runner.kaiming_bound)
    dev = torch.device("cuda", 0)
    st = runner.GpuConvStress(wl, dr.weights[0])
    xd = torch.from_numpy(dr.batches[0][0]).to(dev)
    dd = torch.from_numpy(dr.delta).to(dev)
    g = torch.empty(dd.shape, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    ly = wl.blocks[0].layers[0]
    c, h, w = wl.in_shape
    macs = wl.batch * h * w * ly.c_out * 9 * ly.c_in
    per = []
    st.ctx.kernel_timing(True)
    for r in range(reps):
        lw = limbs_for(int(st.w.abs().max().item()))          # the weights this repeat reads
        w_before = st.w.clone()
        st.ctx.sync()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st.repeat(xd, dd)
        e1.record(stream)
        st.ctx.sync()
        kt = {name: st.ctx.kernel_time(c)[0] for c, name in KERNEL_CLASSES.items()}
        # g of this repeat (for its limb passes) from an untimed replay with g tapped: the same
        # weights in, the same weights out
        w_after = st.w.clone()
        st.w.copy_(w_before)
        st.ctx.kernel_timing(False)
        st.repeat(xd, dd, taps={"g": [g]})
        st.ctx.sync()
        st.ctx.kernel_timing(True)
        if not torch.equal(st.w, w_after):
            raise RuntimeError("stress repeat %d: the replay's weights differ" % r)
        lg = offset_g_limbs(g)
        per.append({"ms": e0.elapsed_time(e1), "kernels_ms": kt,
                    "passes": {"k_conv_tile<fwd>": lw, "k_conv_tile<dx>": lg * lw,
                               "k_conv_dw_planes": lg}})
    st.ctx.kernel_timing(False)

    def summary(rs):
        ms = float(np.median([r["ms"] for r in rs]))
        out = {"repeats": len(rs), "ms_per_repeat": round(ms, 4),
               "algorithmic_TOPs": round(3 * 2 * macs / (ms * 1e-3) / 1e12, 2),
               "frac": round(3 * 2 * macs / (ms * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4), "kernels": {}}
        for name in KERNEL_CLASSES.values():
            kms = float(np.median([r["kernels_ms"][name] for r in rs]))
            passes = int(np.median([r["passes"][name] for r in rs]))
            tops = 2 * macs / (kms * 1e-3) / 1e12 if kms > 0 else 0.0
            out["kernels"][name] = {"ms": round(kms, 4), "algorithmic_TOPs": round(tops, 2),
                                    "frac": round(tops / PEAK_INT8_TOPS, 4), "limb_passes": passes,
                                    "mfma_TOPs": round(tops * passes, 2),
                                    "mfma_frac": round(tops * passes / PEAK_INT8_TOPS, 4)}
        return out

    res = {"workload": wl.name, "repeats": reps, "gop_per_repeat": round(3 * 2 * macs / 1e9, 1),
           "timing": "HIP events around each whole repeat (forward, back-propagation, IntegerSGD); "
                     "kernel times from the kernels' own device timestamps",
           "repeat_1": summary(per[:1])}
    if reps > 1:
        res["steady_state"] = summary(per[1:])
    del st, xd, dd, g
    return res


def paper_nets(steps: int = 10, warmup: int = 2):
    """The paper's own architectures (Tab. 1) at their batch of 64 (Tab. 6) on synthetic CIFAR-10-
    and MNIST-shaped inputs: images/s of the training iteration (HIP events around `steps`
    iterations after `warmup`; graph replay, or eager launches for workloads with dropout, whose
    generator step changes every iteration) and of inference (nitro_net_infer)."""
    import torch
    from paper_2407_11698_amd import runner
    from paper_2407_11698_amd import workloads as WL
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    res = {}
    for wl in WL.PAPER_NETS:
        dr = WL.draw_workload(wl, runner.kaiming_bound, steps=wl.steps)
        xs = [torch.from_numpy(x).to(dev) for x, _ in dr.batches]
        ys = [torch.from_numpy(y).to(dev) for _, y in dr.batches]
        net = runner.GpuNet(wl, dr.weights)
        graph = not (wl.dropout_conv_ppm or wl.dropout_lin_ppm)
        step = net.step_graph if graph else net.step
        if graph:
            for x, y in zip(xs, ys):
                net.prepare_graph(x, y)
        for i in range(warmup):
            step(xs[i % len(xs)], ys[i % len(ys)])
        net.ctx.sync()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(steps):
            step(xs[i % len(xs)], ys[i % len(ys)])
        e1.record(stream)
        net.ctx.sync()
        ms = e0.elapsed_time(e1) / steps
        net.infer(xs[0])
        net.ctx.sync()
        f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        f0.record(stream)
        for i in range(steps):
            net.infer(xs[i % len(xs)])
        f1.record(stream)
        net.ctx.sync()
        ims = f0.elapsed_time(f1) / steps
        res[wl.name] = {"batch": wl.batch, "train_images_per_s": round(wl.batch / (ms * 1e-3), 1),
                        "train_ms_per_step": round(ms, 4), "launch": "graph replay" if graph else "eager",
                        "dropout_ppm": {"conv": wl.dropout_conv_ppm, "linear": wl.dropout_lin_ppm},
                        "infer_images_per_s": round(wl.batch / (ims * 1e-3), 1),
                        "infer_ms_per_batch": round(ims, 4)}
        del net, xs, ys
    return res


def infer_bench(reps: int = 20):
    """Inference (forward and prediction, nitro_net_infer) of the benchmark workload with the
    initial weights, images/s over `reps` batches (HIP events)."""
    import torch
    from paper_2407_11698_amd import runner
    from paper_2407_11698_amd import workloads as WL
    wl = WL.VGG_CNN
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    dr = WL.draw_workload(wl, runner.kaiming_bound, steps=2)
    net = runner.GpuNet(wl, dr.weights)
    x = torch.from_numpy(dr.batches[0][0]).to(dev)
    net.infer(x)
    net.ctx.sync()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        net.infer(x)
    e1.record(stream)
    net.ctx.sync()
    ms = e0.elapsed_time(e1) / reps
    return {"workload": wl.name, "batch": wl.batch, "images_per_s": round(wl.batch / (ms * 1e-3), 1),
            "ms_per_batch": round(ms, 4)}


def preprocess_bench(reps: int = 10):
    """The integer pre-processing of Appendix A on the CIFAR-10-sized synthetic byte dataset
    (50000 x 32 x 32 x 3): device time per pass (HIP events), and HBM rate of its algorithmic
    traffic, 3 bytes per element (the statistics need the data read once, the normalisation
    reads it again and writes it), against the 8 TB/s peak."""
    import torch
    from paper_2407_11698_amd import nitro as N
    from paper_2407_11698_amd import workloads as WL
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    x = torch.from_numpy(WL.draw_image_bytes(WL.CIFAR10_BYTES).reshape(-1)).to(dev)
    out = torch.empty(x.numel(), dtype=torch.int8, device=dev)
    stats = torch.zeros(3, dtype=torch.int64, device=dev)
    ws = torch.empty(N.preprocess_query(x.numel()), dtype=torch.uint8, device=dev)
    ctx = N.Context(0)
    ctx.preprocess(x, out, stats, ws)
    ctx.sync()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        ctx.preprocess(x, out, stats, ws)
    e1.record(stream)
    ctx.sync()
    ms = e0.elapsed_time(e1) / reps
    gbs = 3 * x.numel() / (ms * 1e-3) / 1e9
    st = stats.cpu().tolist()
    ctx.close()
    return {"dataset": "50000x32x32x3 uint8 (synthetic)", "ms": round(ms, 4),
            "algorithmic_bytes": 3 * x.numel(), "GB_per_s": round(gbs, 1),
            "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "mu": st[0], "omega": st[1],
            "clamped": st[2]}


def cpu_baseline(wl, min_s: float = 12.0, budget_s: float = 25.0):
    """The CPU oracle, untuned, on a bounded sample of the same workload: full training
    iterations at a reduced batch (cycling through the ten seeded batches) until at least
    `min_s` seconds have passed; it stops early only past `budget_s`."""
    from oracle import oracle as O
    from paper_2407_11698_amd import workloads as WL
    batch = 16
    sample = WL.scaled(wl, batch)
    dr = WL.draw_workload(sample, O.kaiming_bound, steps=sample.steps)
    hp = O.Hyper(sample.gamma_inv, sample.lambda_inv_fw, sample.lambda_inv_lr, sample.alpha_inv,
                 sample.n_classes)
    net = O.OracleNet([(len(b.layers), b.maxpool, b.learning) for b in sample.blocks],
                      sample.head, dr.weights, hp)
    t0 = time.perf_counter()
    steps = 0
    while True:
        net.train_step(*dr.batches[steps % len(dr.batches)])
        steps += 1
        el = time.perf_counter() - t0
        if el >= min_s or el > budget_s:
            break
    return {"value": round(batch * steps / el, 3), "unit": "images/s", "cores": O.num_threads(),
            "kind": "oracle",
            "sample": "%d training iterations of the same workload at batch %d (%.1f s); "
                      "host %s" % (steps, batch, el, cpu_model())}


ONE_CORE_SRC = """
import sys, time, json
sys.path.insert(0, %r)
from oracle import oracle as O
from paper_2407_11698_amd import workloads as WL
sample = WL.scaled(WL.VGG_CNN, %d)
dr = WL.draw_workload(sample, O.kaiming_bound, steps=sample.steps)
hp = O.Hyper(sample.gamma_inv, sample.lambda_inv_fw, sample.lambda_inv_lr, sample.alpha_inv,
             sample.n_classes)
net = O.OracleNet([(len(b.layers), b.maxpool, b.learning) for b in sample.blocks], sample.head,
                  dr.weights, hp)
t0 = time.perf_counter(); steps = 0
while True:
    net.train_step(*dr.batches[steps %% len(dr.batches)]); steps += 1
    el = time.perf_counter() - t0
    if el >= %f:
        break
print(json.dumps({"steps": steps, "seconds": el, "threads": O.num_threads()}))
"""


def cpu_baseline_one_core(min_s: float = 8.0, batch: int = 4):
    """The CPU oracle on one core (a child process with OMP_NUM_THREADS=1, started before this
    process touches the GPU): training iterations of the benchmark workload at batch `batch`,
    for at least `min_s` seconds."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", ONE_CORE_SRC % (ROOT, batch, min_s)], env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=180)
    if r.returncode != 0:
        return {"error": r.stderr.strip().splitlines()[-1:] or ["exit %d" % r.returncode]}
    d = json.loads(r.stdout.strip().splitlines()[-1])
    return {"value": round(batch * d["steps"] / d["seconds"], 3), "unit": "images/s",
            "cores": d["threads"], "kind": "oracle",
            "sample": "%d training iterations of the same workload at batch %d (%.1f s)"
                      % (d["steps"], batch, d["seconds"])}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch every kernel from the host each step instead of replaying the "
                         "captured iteration (nitro_train_step_graph)")
    ap.add_argument("--serial-steps", type=int, default=9,
                    help="training iterations run after the timed region with every block on "
                         "one stream, for per-launch kernel times without overlap (0 skips)")
    ap.add_argument("--stress-reps", type=int, default=20,
                    help="cumulative repeats of the single conv-layer stress case measured after "
                         "the training iterations (0 skips it)")
    ap.add_argument("--mfma-probe-iters", type=int, default=20000,
                    help="MFMAs per chain of the int8 matrix-core rate probe (0: skip it)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the paper architectures, the inference and the pre-processing "
                         "measurements after the training iterations")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="run one device-to-device copy of this many MiB before the warm-up: "
                         "the known-size reference for hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU only; --gpus %d is not supported" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    # the one-core oracle figure first, in a child process, before this process uses the GPU
    one_core = None if args.no_cpu_baseline else cpu_baseline_one_core()

    import torch
    from paper_2407_11698_amd import nitro as N
    from paper_2407_11698_amd import runner
    from paper_2407_11698_amd import workloads as WL

    wl = WL.VGG_CNN
    dev = torch.device("cuda", 0)
    dr = WL.draw_workload(wl, runner.kaiming_bound)
    graph = not args.eager
    # the library runs on a stream of its own (a captured graph needs a non-default stream);
    # torch's copies below are issued on the same stream, so they are ordered with it
    stream = torch.cuda.Stream(dev)
    torch.cuda.set_stream(stream)
    # the ten seeded batches resident in HBM; with graph replay each has its own captured
    # iteration (prepared before the warm-up), so no input is copied between iterations
    xs = [torch.from_numpy(x).to(dev) for x, _ in dr.batches]
    ys = [torch.from_numpy(y).to(dev) for _, y in dr.batches]
    net = runner.GpuNet(wl, dr.weights)
    w0 = net.w_flat.clone()              # every weight, restored with one copy every ten steps
    period = len(xs)

    def prepare():
        for x, y in zip(xs, ys):
            net.prepare_graph(x, y)

    def run(k0, k):
        for i in range(k0, k0 + k):
            if i % period == 0:
                net.w_flat.copy_(w0)
            if graph:
                net.step_graph(xs[i % period], ys[i % period])
            else:
                net.step(xs[i % period], ys[i % period])

    if args.copy_mib > 0:
        src = torch.zeros(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # per-kernel timing is switched on before the warm-up: the graph is captured once, with its
    # timing events, outside the timed region (the events then hold the last replay's times)
    warmup = max(args.warmup, 1) if graph else args.warmup
    if graph:
        net.ctx.kernel_timing(True)
        prepare()
    run(0, warmup)
    net.ctx.sync()
    if not graph:
        net.ctx.kernel_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(warmup, args.steps)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    net.ctx.sync()                        # raises if any kernel flagged overflow or a bad label
    ktime = {KERNEL_CLASSES[c]: net.ctx.kernel_time(c) for c in KERNEL_CLASSES}
    net.ctx.kernel_timing(False)
    timed_steps = 1 if graph else args.steps    # graph: the events of the last replay

    # per-iteration times (median and min), after the timed region: events on the library's
    # stream around each iteration of the same sequence
    if graph:
        prepare()                         # the graphs again, now captured without timing
        run(warmup, 1)
    per_step = []
    for i in range(args.steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        run(warmup + i, 1)
        e1.record(stream)
        per_step.append((e0, e1))
    torch.cuda.synchronize()
    step_ms = sorted(a.elapsed_time(b) for a, b in per_step)
    net.ctx.sync()

    ops = conv_layer_ops(wl)
    per_class = {}
    for name, (ms, launches) in ktime.items():
        tops = ops[name] * timed_steps / (ms * 1e-3) / 1e12 if ms > 0 else 0.0
        per_class[name] = {"ms_per_step": round(ms / timed_steps, 4), "launches": launches,
                           "avg_launch_us": round(ms * 1e3 / launches, 2) if launches else None,
                           "algorithmic_TOPs": round(tops, 3)}
    dom = max(per_class, key=lambda k: per_class[k]["ms_per_step"])
    achieved = per_class[dom]["algorithmic_TOPs"]

    # the roofline kernel's launch durations: the same trajectory after the timed region, launched
    # eagerly with every block on the library's one stream (a launch then has the GPU to itself,
    # as under a kernel-trace profiler), each launch of a timed kernel class measured by the
    # device timestamps its workgroups record (first start to last end); then the same with HIP
    # events around each launch on its stream, as a cross-check (the event markers add a few
    # microseconds per launch)
    serial, serial_ev = {}, {}
    if args.serial_steps > 0:
        net.ctx.set_aux_streams(0)
        for res, events in ((serial, False), (serial_ev, True)):
            net.w_flat.copy_(w0)
            net.step(xs[0], ys[0])
            net.ctx.sync()
            net.ctx.kernel_timing(True, events=events)
            for i in range(1, 1 + args.serial_steps):
                net.step(xs[i % period], ys[i % period])
            net.ctx.sync()
            for c, name in KERNEL_CLASSES.items():
                ms, launches = net.ctx.kernel_time(c)
                if launches:
                    res[name] = {"ms_per_step": round(ms / args.serial_steps, 4),
                                 "launches_per_step": launches // args.serial_steps,
                                 "avg_launch_us": round(ms * 1e3 / launches, 2),
                                 "algorithmic_TOPs": round(ops[name] * args.serial_steps / (ms * 1e-3) / 1e12, 3)}
            net.ctx.kernel_timing(False)
        net.ctx.set_aux_streams(3)
    conv_ms = sum(v["ms_per_step"] for v in per_class.values())
    conv_tops = sum(ops.values()) / (conv_ms * 1e-3) / 1e12 if conv_ms > 0 else 0.0

    out = {
        "metric": "images/s per IntegerSGD training step; int8 conv TOPS as % of MFMA peak",
        "value": round(wl.batch * args.steps / el, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmup,
        "ms_per_step": round(el * 1e3 / args.steps, 4),
        "step_ms": {"median": round(step_ms[len(step_ms) // 2], 4), "min": round(step_ms[0], 4),
                    "iterations": len(step_ms), "timing": "HIP events around each iteration, "
                                                          "after the timed region"},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "input": "3x32x32 int8",
                   "blocks": "conv 3-64-64, 64-128-128, 128-256-256, 256-512-512, pool, "
                             "learning layer to 100 classes", "gamma_inv": wl.gamma_inv,
                   "lambda_inv_fw": wl.lambda_inv_fw, "lambda_inv_lr": wl.lambda_inv_lr,
                   "alpha_inv": wl.alpha_inv, "rounding": "floor",
                   "launch": "graph replay" if graph else "eager"},
        "conv_mfma": {"algorithmic_TOPs": round(conv_tops, 3),
                      "frac_of_int8_peak": round(conv_tops / PEAK_INT8_TOPS, 5),
                      "timed_region_per_kernel": per_class,
                      "timed_region_timing": "device timestamps of each launch's first and last "
                                             "workgroups, inside the replayed graph (blocks on "
                                             "four streams)"},
    }
    if serial_ev:
        # the dominant kernel class of the serial pass; achieved = its algorithmic ops per step /
        # its summed launch time per step (= ops per launch / average launch duration), the
        # launches timed by HIP events on their stream (what a kernel trace of the same command
        # reports as their durations); the kernels' own device timestamps beside it
        sdom = max(serial_ev, key=lambda k: serial_ev[k]["ms_per_step"])
        sd = serial_ev[sdom]
        out["roofline"] = {"bound": "mfma", "kernel": sdom, "achieved": sd["algorithmic_TOPs"],
                           "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                           "frac": round(sd["algorithmic_TOPs"] / PEAK_INT8_TOPS, 5),
                           "avg_launch_us": sd["avg_launch_us"],
                           "launches_per_step": sd["launches_per_step"],
                           "ops_per_step": ops[sdom],
                           "traffic": recorded_traffic(sdom),
                           "avg_launch_us_device_timestamps": serial.get(sdom, {}).get("avg_launch_us"),
                           "timing": "HIP events around each launch on the stream it is launched "
                                     "on, %d eager iterations of the same trajectory after the "
                                     "timed region, every block on one stream; "
                                     "avg_launch_us_device_timestamps: the launches' first "
                                     "workgroup start to last workgroup end (s_memrealtime) in "
                                     "the same setting" % args.serial_steps}
        out["conv_mfma"]["serial_per_kernel"] = serial
        out["conv_mfma"]["serial_per_kernel_events"] = serial_ev
    else:
        out["roofline"] = {"bound": "mfma", "kernel": dom, "achieved": achieved,
                           "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                           "frac": round(achieved / PEAK_INT8_TOPS, 5),
                           "traffic": recorded_traffic(dom),
                           "timing": "device timestamps in the timed region"}
    if args.mfma_probe_iters > 0:
        # the dense int8 matrix-core rate on this GPU (register-only MFMA chains, two waves per
        # SIMD); `peak` above stays the published figure
        out["mfma_rate_probe"] = {"TOPs": round(net.ctx.mfma_rate(2, args.mfma_probe_iters), 1),
                                  "waves_per_simd": 2, "published_TOPs": PEAK_INT8_TOPS}
    if args.stress_reps > 0:
        out["stress_conv"] = stress_layer(args.stress_reps)
    if not args.no_extras:
        out["paper_nets"] = paper_nets()
        out["inference"] = infer_bench()
        out["preprocess"] = preprocess_bench()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
        out["cpu_baseline"]["one_core"] = one_core
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
