"""Benchmark of the Two-Bit Networks hot path on one MI355X.

One step = one pass of the whole hot path over one batch (Algorithm 1 on one large
layer): quantise the real weights (Sec. 2 Eq. 3-5) -> forward (Eq. 1) -> backward to the
input and to the approximate filter (Sec. 3) -> SGD update of the real weights (Sec. 4).
Workload: conv 3x3, 256 -> 256 channels, 56 x 56, pad 1, batch 128, bf16 activations
N(0,1), upstream gradient N(0,1), real weights N(0, 0.05^2), lr 0.1, momentum 0.9, weight
decay 1e-4.  Inputs are seeded synthetic tensors already resident in HBM.

Prints one JSON line: the effective TFLOP/s of the step (2 FLOP per multiply-add of the
three dense contractions, the count of the full-precision layer), the roofline of the
dominant kernel (timed live with HIP events on the stream it runs on), and the fp64 CPU
oracle timed on a bounded slice of the same step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_INT8_TOPS = 5000.0     # MI355X dense int8 MFMA
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA

LAYER = dict(n=128, h=56, w=56, c=256, k=256, r=3, s=3, stride=1, pad=1)
LR, MOMENTUM, WD = 0.1, 0.9, 1e-4


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warmup-seconds", type=float, default=0.3,
                    help="keep running untimed steps until at least this much time has passed "
                         "(the GPU clocks rise over the first tens of milliseconds of load)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-resnet", action="store_true", help="skip the ResNet-18 forward figures")
    ap.add_argument("--no-small", action="store_true", help="skip the single-layer, LeNet and VGG figures")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="budget of the oracle's training-step sample")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain device copy of known size (HBM counter calibration)")
    ap.add_argument("--only", choices=["resnet", "single", "lenet", "vgg", "ws", "int8", "fp8", "fused"],
                    help="profiling aid: run just this workload (no training step, no contract line)")
    return ap.parse_args()


def layer_flops():
    """FLOP of one dense contraction of the layer (2 per multiply-add)."""
    L = LAYER
    P = (L["h"] + 2 * L["pad"] - L["r"]) // L["stride"] + 1
    Q = (L["w"] + 2 * L["pad"] - L["s"]) // L["stride"] + 1
    M = L["n"] * P * Q
    kred = L["r"] * L["s"] * L["c"]
    return 2.0 * M * L["k"] * kred, P, Q


# Which kernel carries each timed call, and the sources its HBM counters were taken on.
KERNEL_OF_OP = {
    "fwd": ("conv_dma_kernel<128, 256, 1, 4, 3, false, true, 1>", ["tbn_conv_dma.hip", "tbn_dma.h", "tbn_device.h"]),
    "bwd_data": ("conv_dma_kernel<128, 256, 1, 4, 3, true, true, 1>", ["tbn_conv_dma.hip", "tbn_dma.h", "tbn_device.h"]),
    "bwd_weight": ("wgrad_rows_kernel", ["tbn_wgrad_dma.hip", "tbn_dma.h", "tbn_device.h"]),
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "conv3x3_256x256_56x56_b128_train_step_traffic.json")


def measured_traffic(op):
    """Calibrated HBM bytes per launch from the committed counter run, or None when the
    kernel source changed since the counters were taken."""
    import hashlib
    try:
        data = json.load(open(TRAFFIC_FILE))
    except OSError:
        return None
    key, files = KERNEL_OF_OP[op]
    m = hashlib.sha256()
    for f in files:
        m.update(open(os.path.join(ROOT, "paper_1701_00485_amd", "csrc", f), "rb").read())
    for name, rec in data["kernels"].items():
        if key in name and rec["source_sha"] == m.hexdigest()[:16]:
            return rec["bytes"]
    return None


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(budget_s: float):
    """The fp64 oracle (plain loops, OpenMP over the host cores) timed on the workloads, in
    the same run as the GPU:
      * the training step (the headline workload): quantise and SGD over the whole layer,
        the three convolutions on as many images of the batch as fit in `budget_s` seconds
        (at least one; the work is linear in the batch, so the mean per-image time is
        scaled by 128);
      * the single layer (16 x 28 x 28 x 1 -> 32 filters 5x5), whole, on one thread and on
        all cores (median of several calls);
      * one whole LeNet training iteration at batch 256;
      * VGG-small training iterations on a slice of 4 images of the batch of 128, scaled
        by 32 (the contractions are linear in the batch).
    `value` is the training step's rate, in the metric's unit."""
    import oracle
    import synth
    from oracle import nets

    L = LAYER
    threads = len(os.sched_getaffinity(0))
    oracle.set_threads(threads)
    d = oracle.ConvDesc(1, L["h"], L["w"], L["c"], L["k"], L["r"], L["s"], L["stride"], L["pad"])
    P, Q = d.out_dims()
    n = L["r"] * L["s"] * L["c"]
    w = synth.normal(5, "w", (L["k"], n), 0.05)
    v = np.zeros_like(w)
    t0 = time.perf_counter()
    q = oracle.quantize(w)
    a64 = q.alpha.astype(np.float64)
    t_quant = time.perf_counter() - t0
    conv_s, images, g = 0.0, 0, None
    while images < L["n"] and (images == 0 or conv_s < budget_s):
        x = oracle.bf16_bits_to_f64(synth.normal_bf16(5, "x1_%d" % images, (1, L["h"], L["w"], L["c"])))
        dy = oracle.bf16_bits_to_f64(synth.normal_bf16(5, "dy1_%d" % images, (1, P, Q, L["k"])))
        t1 = time.perf_counter()
        oracle.conv_fwd(d, x, q.codes, a64)
        oracle.conv_bwd_data(d, dy, q.codes, a64)
        g = oracle.conv_bwd_weight(d, x, dy).reshape(L["k"], n)
        conv_s += time.perf_counter() - t1
        images += 1
    t2 = time.perf_counter()
    oracle.sgd(w, v, g, LR, MOMENTUM, WD)
    t_sgd = time.perf_counter() - t2
    step_s = t_quant + t_sgd + conv_s / images * L["n"]
    conv_flops, _, _ = layer_flops()
    out = {
        "value": round(3 * conv_flops / step_s / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "affinity_cores": threads,
        "cpu_model": _cpu_model(),
        "kind": "oracle",
        "sample": "fp64 oracle: quantise + SGD over the full 256x3x3x256 layer, fwd/bwd_data/bwd_weight "
                  "on %d of 128 images (mean per image scaled x128); measured %.1f s, extrapolated %.0f s "
                  "per step" % (images, t_quant + t_sgd + conv_s, step_s),
    }
    configs = {"train_step_s": round(step_s, 2)}

    # single layer, whole: one thread and all cores
    d1 = oracle.ConvDesc(16, 28, 28, 1, 32, 5, 5, 1, 2)
    x1 = oracle.round_bf16(synth.uniform(1, "x", (16, 28, 28, 1)))
    q1 = oracle.quantize(synth.normal(1, "w", (32, 25), 0.05))
    a1 = q1.alpha.astype(np.float64)
    fl1 = 2.0 * 16 * 28 * 28 * 32 * 25
    for label, nthr in (("single_thread", 1), ("all_cores", threads)):
        oracle.set_threads(nthr)
        ts = []
        for _ in range(7):
            t = time.perf_counter()
            oracle.conv_fwd(d1, x1, q1.codes, a1)
            ts.append(time.perf_counter() - t)
        med = float(np.median(ts))
        configs["single_layer_fwd_" + label] = {"us_per_call": round(med * 1e6, 1), "threads": nthr,
                                               "tflops": round(fl1 / med / 1e12, 6)}
    oracle.set_threads(threads)

    # LeNet: one whole training iteration at batch 256
    from paper_1701_00485_amd.networks import LeNet, VGGSmall
    xl = oracle.bf16_bits_to_f64(synth.bf16_bits(synth.uniform(2, "bench_x", (256, 28, 28, 1))))
    lab = synth.labels(2, "bench_lab", 256, 10)
    wl = {name: synth.normal(2, name, (cout, k * k * cin), 0.05) for name, cin, cout, k, *_ in nets.LENET}
    vl = {name: np.zeros(wv.shape) for name, wv in wl.items()}
    t = time.perf_counter()
    nets.lenet_iteration(xl, lab, wl, vl, LR)
    t_lenet = time.perf_counter() - t
    configs["lenet_iteration"] = {"s": round(t_lenet, 3), "images_per_s": round(256 / t_lenet, 1),
                                  "tflops": round(LeNet.train_flops(256) / t_lenet / 1e12, 6), "batch": 256}

    # VGG-small: iterations on 4 images, scaled to the batch of 128
    nv = 4
    xv = oracle.bf16_bits_to_f64(synth.normal_bf16(3, "bench_x", (nv, 32, 32, 3)))
    labv = synth.labels(3, "bench_lab", nv, 10)
    wv = {name: synth.normal(3, name, (cout, 9 * cin), 0.05) for name, cin, cout, _ in nets.VGG}
    wv["fc"] = synth.normal(3, "fc", (10, 16 * 512), 0.05)
    vv = {name: np.zeros(a.shape) for name, a in wv.items()}
    bn = {name: (np.ones(cout), np.zeros(cout)) for name, _, cout, _ in nets.VGG}
    bnv = {name: (np.zeros(cout), np.zeros(cout)) for name, _, cout, _ in nets.VGG}
    t = time.perf_counter()
    nets.vgg_iteration(xv, labv, wv, vv, bn, bnv, LR)
    t_vgg = (time.perf_counter() - t) * (128 / nv)
    configs["vgg_small_iteration"] = {"s": round(t_vgg, 2), "images_per_s": round(128 / t_vgg, 2),
                                      "tflops": round(VGGSmall.train_flops(128) / t_vgg / 1e12, 6), "batch": 128,
                                      "sample": "%d of 128 images, time scaled x%d" % (nv, 128 // nv)}
    out["configs"] = configs
    return out


def resnet18_fwd(dev, steps=10, warmup=3):
    """ResNet-18 forward (all convolutions and the classifier two-bit) at batch 64 and 1:
    images/s, and the achieved TFLOP/s of the nine stride-1 3x3 layers with C = K >= 128."""
    import torch

    import synth
    from paper_1701_00485_amd.networks import ResNet18

    net = ResNet18(device=dev)
    out = {"model": "ResNet-18, two-bit convolutions and classifier, BN folded, 224x224 bf16 N(0,1)"}
    stream = torch.cuda.current_stream()
    for batch in (64, 1):
        x = torch.from_numpy(synth.normal_bf16(4, "bench_x%d" % batch, (batch, 224, 224, 3)).view(np.int16))
        x = x.to(dev).view(torch.bfloat16)
        for _ in range(warmup):
            net.forward(x)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            net.forward(x)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        rec = {"ms_per_batch": round(ms, 4), "images_per_s": round(batch / (ms * 1e-3), 1),
               "effective_tflops": round(ResNet18.flops(batch) / (ms * 1e-3) / 1e12, 2)}
        if batch == 1:
            # the whole forward captured once as a HIP graph and replayed
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(stream)
            with torch.cuda.stream(side):
                net.forward(x)
                torch.cuda.synchronize()
                with torch.cuda.graph(g, stream=side):
                    logits_g = net.forward(x)
            torch.cuda.synchronize()
            for _ in range(warmup):
                g.replay()
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(steps * 10):
                g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            gms = e0.elapsed_time(e1) / (steps * 10)
            rec["graph_ms_per_batch"] = round(gms, 4)
            rec["graph_images_per_s"] = round(1.0 / (gms * 1e-3), 1)
            del logits_g
        out["batch%d" % batch] = rec
    # the nine large stride-1 3x3 layers at batch 64, each timed alone
    x = torch.from_numpy(synth.normal_bf16(4, "bench_x64", (64, 224, 224, 3)).view(np.int16)).to(dev)
    trace = []
    net.forward(x.view(torch.bfloat16), trace)
    torch.cuda.synchronize()
    layers = []
    for kind, layer, inp, outp, res in trace:
        if kind != "conv" or layer.k != 3 or layer.stride != 1 or layer.cin < 128:
            continue
        relu = True
        # the calls are captured as a HIP graph and replayed, so the time is the device's
        # (a layer of ~15 GFLOP is shorter than the host's per-call work)
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            for _ in range(2):
                layer(inp, relu=relu, residual=res)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=side):
                for _ in range(steps):
                    layer(inp, relu=relu, residual=res)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        reps = []  # median of five timed replays
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            graph.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            reps.append(e0.elapsed_time(e1) / steps * 1e3)
        us = float(np.median(reps))
        del graph
        n, h, w, c = inp.shape
        fl = 2.0 * n * h * w * layer.cout * 9 * c
        layers.append({"layer": layer.name, "us": round(us, 1), "tflops": round(fl / (us * 1e-6) / 1e12, 1)})
    fr = [l["tflops"] / PEAK_BF16_TFLOPS for l in layers]
    out["large_3x3_layers_batch64"] = layers
    out["large_3x3_frac_of_bf16_peak"] = {"min": round(min(fr), 4), "mean": round(float(np.mean(fr)), 4)}
    return out


def small_configs(dev, steps=20, warmup=3, which=("single", "lenet", "vgg")):
    """The smaller workloads: one two-bit layer on MNIST-shaped fp32 input (forward only,
    latency-bound), and full training iterations of the MNIST-shaped LeNet (batch 256) and
    the CIFAR-shaped VGG (batch 128)."""
    import torch

    import paper_1701_00485_amd as tbn
    import synth
    from paper_1701_00485_amd.networks import LeNet, VGGSmall

    stream = torch.cuda.current_stream()
    out = {}

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    # single layer: 16 x 28 x 28 x 1 fp32 U[0,1) -> 32 filters 5x5 pad 2, fp32 output
    if "single" in which:
        _single_layer(dev, out, timed)
    for name, cls, batch, mk in (
            ("lenet_train", LeNet, 256,
             lambda: synth.bf16_bits(synth.uniform(2, "bench_x", (256, 28, 28, 1)))),
            ("vgg_small_train", VGGSmall, 128, lambda: synth.normal_bf16(3, "bench_x", (128, 32, 32, 3)))):
        if name.split("_")[0] not in which:
            continue
        _net_train(dev, out, timed, name, cls, batch, mk, steps)
    return out


def _single_layer(dev, out, timed):
    import torch

    import paper_1701_00485_amd as tbn
    import synth

    d = tbn.ConvDesc(16, 28, 28, 1, 32, 5, 5, 1, 2)
    x = torch.from_numpy(synth.uniform(1, "x", (16, 28, 28, 1))).to(dev)
    w = torch.from_numpy(synth.normal(1, "w", (32, 25), 0.05)).to(dev)
    codes, alpha, _ = tbn.quantize(w, want_counts=False)
    y = torch.empty((16, 28, 28, 32), dtype=torch.float32, device=dev)
    eager_ms = timed(lambda: tbn.conv2d_fwd(d, x, codes, alpha, y=y), 200)
    # device time per call: 200 calls captured once as a HIP graph and replayed (the eager
    # figure above includes the host-side argument checks and launch of every call)
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for _ in range(200):
            tbn.conv2d_fwd(d, x, codes, alpha, y=y)
    torch.cuda.synchronize()
    ms = timed(graph.replay, 5) / 200
    fl = 2.0 * 16 * 28 * 28 * 32 * 25
    byts = 16 * 28 * 28 * 4 + y.numel() * 4 + codes.numel() * 4 + 32 * 4
    out["single_layer_fwd"] = {"shape": "16x28x28x1 fp32 -> 32 filters 5x5 pad 2, fp32 out", "us_per_call": round(ms * 1e3, 2),
                               "timing": "graph replay of 200 calls (device time per call)",
                               "eager_us_per_call": round(eager_ms * 1e3, 2),
                               "effective_tflops": round(fl / (ms * 1e-3) / 1e12, 3),
                               "hbm_frac": round(byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}


def _net_train(dev, out, timed, name, cls, batch, mk, steps):
    import torch

    import synth

    stream = torch.cuda.current_stream()
    net = cls(device=dev)
    xb = torch.from_numpy(mk().view(np.int16)).to(dev).view(torch.bfloat16)
    lab = torch.from_numpy(synth.labels(2, "bench_lab", batch, 10).astype(np.int32)).to(dev)
    ms = timed(lambda: net.step(xb, lab), steps)
    # the same iteration captured once as a HIP graph and replayed (no host launch work)
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        net.step(xb, lab)
    torch.cuda.synchronize()
    gms = timed(graph.replay, steps)
    # the update fused with the next iteration's quantisation (one pass over the real
    # weights; the iteration then has no separate quantisation), eager and as a graph
    fms = timed(lambda: net.step(xb, lab, fused=True), steps)
    fgraph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(fgraph, stream=side):
        net.step(xb, lab, fused=True)
    torch.cuda.synchronize()
    fgms = timed(fgraph.replay, steps)
    out[name] = {"batch": batch, "ms_per_iteration": round(ms, 4), "images_per_s": round(batch / (ms * 1e-3), 1),
                 "effective_tflops": round(cls.train_flops(batch) / (ms * 1e-3) / 1e12, 2),
                 "graph_ms_per_iteration": round(gms, 4),
                 "graph_images_per_s": round(batch / (gms * 1e-3), 1),
                 "fused_update_ms_per_iteration": round(fms, 4),
                 "fused_update_graph_ms_per_iteration": round(fgms, 4)}


def weight_streaming(dev, sets=8, reps=20):
    """Batch-1 fully-connected layer 8192 -> 32768 (67 MB of packed codes) cycled over 8
    filter sets (537 MB, more than the 256 MB last-level cache), so every call streams its
    codes from HBM: achieved GB/s of the algorithmic bytes (codes, scales, input, output)."""
    import torch

    import paper_1701_00485_amd as tbn

    C, K = 8192, 32768
    d = tbn.ConvDesc(1, 1, 1, C, K, 1, 1, 1, 0)
    g = torch.Generator(device=dev)
    g.manual_seed(1701_00485)
    filters = []
    for _ in range(sets):
        w = torch.randn(K, C, device=dev, generator=g) * 0.05  # real filters N(0, 0.05^2)
        codes, alpha, _ = tbn.quantize(w, want_counts=False)
        del w
        filters.append((codes, alpha))
    x = (torch.randn(1, 1, 1, C, device=dev, generator=g)).to(torch.bfloat16)
    y = torch.empty(1, 1, 1, K, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    for _ in range(2):
        for c, a in filters:
            tbn.conv2d_fwd(d, x, c, a, y=y, out_dtype=torch.float32)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        for c, a in filters:
            tbn.conv2d_fwd(d, x, c, a, y=y, out_dtype=torch.float32)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / (reps * sets) * 1e3
    byts = filters[0][0].numel() * 4 + K * 4 + C * 2 + K * 4
    gbs = byts / (us * 1e-6) / 1e9
    return {"shape": "batch 1, 8192 -> 32768, 8 filter sets (537 MB of codes)", "us_per_call": round(us, 2),
            "bytes_per_call": byts, "achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}


def fused_update(dev, reps=20):
    """The update step fused with the next quantisation (one pass over the real weights:
    12 B read + 8.25 B written per weight) against SGD followed by a separate quantisation
    (16 B read + 8.25 B written), on the training layer and on a 4096 x 4608 filter set
    (18.9 M weights, larger than the last-level cache); also the stochastic discretisation
    (weights and uniform numbers read, 8 B, codes written, 0.25 B per weight)."""
    import torch

    import paper_1701_00485_amd as tbn

    stream = torch.cuda.current_stream()
    out = {}
    for name, K, n in (("train_layer_256x2304", 256, 2304), ("filters_4096x4608", 4096, 4608)):
        g = torch.Generator(device=dev)
        g.manual_seed(1701_00485)
        w = torch.randn(K, n, device=dev, generator=g) * 0.05
        v = torch.zeros_like(w)
        gr = torch.randn(K, n, device=dev, generator=g)
        codes, alpha, _ = tbn.quantize(w, want_counts=False)

        def fused():
            tbn.sgd_step_quantize(w, v, gr, 1e-6, 0.9, 1e-4, codes=codes, alpha=alpha, want_counts=False)

        def separate():
            tbn.sgd_step(w, v, gr, 1e-6, 0.9, 1e-4)
            tbn.quantize(w, codes, alpha, want_counts=False)

        uni = torch.rand(K, n, device=dev, generator=g)

        def stochastic():
            tbn.quantize_variant(w, 1.0, uni, codes=codes, alpha=alpha, want_counts=False)

        rec = {}
        for label, fn, byts in (("fused", fused, 20.25), ("separate", separate, 24.25),
                                ("stochastic_quantize", stochastic, 8.25)):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / reps * 1e3
            gbs = byts * K * n / (us * 1e-6) / 1e9
            rec[label] = {"us": round(us, 2), "achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
        out[name] = rec
    return out


def int8_forward(dev, desc, x, codes, alpha, conv_flops, reps=20):
    """The integer-activation variant of the forward pass on the training layer: activation
    codes (2 B read + 1 B written per activation) and the forward pass on the int8 matrix
    cores, timed with HIP events on the stream they run on.  The activation scale is fixed
    once from max|x| (a calibration step, outside the timed region)."""
    import torch

    import paper_1701_00485_amd as tbn

    stream = torch.cuda.current_stream()
    amax = float(x.float().abs().max())
    x_scale = amax / 127.0
    xq = torch.empty(x.shape, dtype=torch.int8, device=dev)
    P, Q = desc.out_dims()
    y = torch.empty((desc.n, P, Q, desc.k), dtype=torch.bfloat16, device=dev)

    def quant():
        tbn.quantize_act_i8(x, 127.0 / amax, q=xq)

    def conv():
        tbn.conv2d_fwd_i8(desc, xq, codes, alpha, x_scale, y=y)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    us_q = timed(quant)
    us_c = timed(conv)
    tops = conv_flops / (us_c * 1e-6) / 1e12
    gbs = 3.0 * x.numel() / (us_q * 1e-6) / 1e9
    return {
        "shape": "conv3x3 256->256 ch, 56x56, pad 1, batch 128; int8 activations, bf16 output",
        "act_quantize": {"us": round(us_q, 2), "achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)},
        "conv_fwd_i8": {"us": round(us_c, 2), "achieved_TOPS": round(tops, 1), "peak_TOPS": PEAK_INT8_TOPS,
                        "frac": round(tops / PEAK_INT8_TOPS, 4)},
    }


def fp8_forward(dev, desc, x, codes, alpha, conv_flops, reps=20):
    """The fp8-activation variant of the forward pass on the training layer: E4M3 activation
    codes (2 B read + 1 B written per activation) and the forward pass on the scaled fp8 x
    fp4 matrix cores, timed with HIP events on the stream they run on.  The activation scale
    is fixed once from max|x| and the filter codes are repacked into the E2M1 layout once
    (calibration and a once-per-weight-update step, outside the timed region)."""
    import torch

    import paper_1701_00485_amd as tbn

    stream = torch.cuda.current_stream()
    amax = float(x.float().abs().max())
    x_scale = amax / 448.0
    xq = torch.empty(x.shape, dtype=torch.uint8, device=dev)
    f4 = tbn.repack_codes_fp4(codes)
    P, Q = desc.out_dims()
    y = torch.empty((desc.n, P, Q, desc.k), dtype=torch.bfloat16, device=dev)

    def quant():
        tbn.quantize_act_fp8(x, 448.0 / amax, q=xq)

    def conv():
        tbn.conv2d_fwd_fp8(desc, xq, f4, alpha, x_scale, y=y)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    us_q = timed(quant)
    us_c = timed(conv)
    tf = conv_flops / (us_c * 1e-6) / 1e12
    gbs = 3.0 * x.numel() / (us_q * 1e-6) / 1e9
    return {
        "shape": "conv3x3 256->256 ch, 56x56, pad 1, batch 128; E4M3 activations x E2M1 two-bit codes, bf16 output",
        "act_quantize": {"us": round(us_q, 2), "achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)},
        "conv_fwd_fp8": {"us": round(us_c, 2), "achieved_TFLOPS": round(tf, 1), "peak_TFLOPS": PEAK_FP8_TFLOPS,
                         "frac": round(tf / PEAK_FP8_TFLOPS, 4)},
    }


def _only(section, dev):
    """One workload alone (for kernel traces and counters of that workload)."""
    if section == "resnet":
        return resnet18_fwd(dev)
    if section in ("single", "lenet", "vgg"):
        return small_configs(dev, which=(section,))
    if section == "ws":
        return weight_streaming(dev)
    if section == "fused":
        return fused_update(dev)
    import torch

    import paper_1701_00485_amd as tbn
    import synth
    L = LAYER
    conv_flops, P, Q = layer_flops()
    desc = tbn.ConvDesc(L["n"], L["h"], L["w"], L["c"], L["k"], L["r"], L["s"], L["stride"], L["pad"])
    x = torch.from_numpy(synth.normal_bf16(5, "x", (L["n"], L["h"], L["w"], L["c"])).view(np.int16)).to(dev)
    w = torch.from_numpy(synth.normal(5, "w", (L["k"], L["r"] * L["s"] * L["c"]), 0.05)).to(dev)
    codes, alpha, _ = tbn.quantize(w, want_counts=False)
    if section == "fp8":
        return fp8_forward(dev, desc, x.view(torch.bfloat16), codes, alpha, conv_flops)
    return int8_forward(dev, desc, x.view(torch.bfloat16), codes, alpha, conv_flops)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (got --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1701_00485_amd as tbn
    import synth

    tbn.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.only:
        print(json.dumps({"only": args.only, "result": _only(args.only, dev)}), flush=True)
        return
    L = LAYER
    conv_flops, P, Q = layer_flops()
    flops = 3 * conv_flops  # forward, backward-data and backward-weight contractions
    n = L["r"] * L["s"] * L["c"]
    desc = tbn.ConvDesc(L["n"], L["h"], L["w"], L["c"], L["k"], L["r"], L["s"], L["stride"], L["pad"])

    def dev_bf16(bits):
        return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)

    x = dev_bf16(synth.normal_bf16(5, "x", (L["n"], L["h"], L["w"], L["c"])))
    dy = dev_bf16(synth.normal_bf16(5, "dy", (L["n"], P, Q, L["k"])))
    w = torch.from_numpy(synth.normal(5, "w", (L["k"], n), 0.05)).to(dev)
    v = torch.zeros_like(w)
    codes = torch.empty(tbn.packed_words(L["k"], n), dtype=torch.int32, device=dev)
    alpha = torch.empty(L["k"], dtype=torch.float32, device=dev)
    y = torch.empty((L["n"], P, Q, L["k"]), dtype=torch.bfloat16, device=dev)
    dx = torch.empty_like(x)
    dw = torch.empty((L["k"], L["r"], L["s"], L["c"]), dtype=torch.float32, device=dev)
    ws_bd = tbn.workspace(tbn.OP_BWD_DATA, desc, dev)
    ws_bw = tbn.workspace(tbn.OP_BWD_WEIGHT, desc, dev)
    stream = torch.cuda.current_stream()

    names = ["quantize", "fwd", "bwd_data", "bwd_weight", "sgd"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record(stream)
        mark(0)
        tbn.quantize(w, codes, alpha, want_counts=False)
        mark(1)
        tbn.conv2d_fwd(desc, x, codes, alpha, y=y)
        mark(2)
        tbn.conv2d_bwd_data(desc, dy, codes, alpha, dx=dx, ws=ws_bd)
        mark(3)
        tbn.conv2d_bwd_weight(desc, x, dy, dw=dw, ws=ws_bw)
        mark(4)
        tbn.sgd_step(w, v, dw, LR, MOMENTUM, WD)
        mark(5)

    # untimed: at least W steps and at least --warmup-seconds of steady load
    warm_run = 0
    t_warm = time.perf_counter()
    while warm_run < args.warmup or time.perf_counter() - t_warm < args.warmup_seconds:
        step()
        torch.cuda.synchronize()
        warm_run += 1
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step(events[i])
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    per_call = {nm: [events[i][j].elapsed_time(events[i][j + 1]) for i in range(args.steps)]
                for j, nm in enumerate(names)}
    per_kernel = {nm: float(np.median(v_)) for nm, v_ in per_call.items()}
    step_times = [events[i][0].elapsed_time(events[i][5]) for i in range(args.steps)]

    if args.copy_probe:
        a = torch.empty(256 * 1024 * 1024, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    conv_names = ["fwd", "bwd_data", "bwd_weight"]
    dom = max(conv_names, key=lambda nm: per_kernel[nm])
    achieved = conv_flops / (per_kernel[dom] * 1e-3) / 1e12
    result = {
        "metric": "2-bit-weight conv effective TFLOP/s + ResNet-18-shape fwd images/sec, 1 GPU",
        "value": round(flops / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm_run,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_median": round(float(np.median(step_times)), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations and gradients, N(0,0.05^2) real weights)",
        "config": {
            "workload": "two-bit conv3x3 training step: quantise -> fwd -> bwd_data -> bwd_weight -> SGD, "
                        "256->256 ch, 56x56, pad 1, batch 128",
            "global_batch": L["n"],
            "flop_per_step": flops,
            "parallelism": "none (1 GPU)",
        },
        "per_kernel_ms": {k: round(v_, 4) for k, v_ in per_kernel.items()},
        "per_kernel_ms_min_max": {k: [round(min(v_), 4), round(max(v_), 4)] for k, v_ in per_call.items()},
        "timing": "per-kernel and per-step figures are medians over the timed steps (HIP events on the "
                  "stream the kernels run on); ms_per_step is the timed region divided by the steps",
        "roofline": {
            "bound": "mfma",
            "kernel": dom,
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic(dom),
        },
    }
    result["int8_forward"] = int8_forward(dev, desc, x, codes, alpha, conv_flops)
    result["int8_forward"]["bf16_fwd_us"] = round(per_kernel["fwd"] * 1e3, 2)
    result["fp8_forward"] = fp8_forward(dev, desc, x, codes, alpha, conv_flops)
    result["fp8_forward"]["bf16_fwd_us"] = round(per_kernel["fwd"] * 1e3, 2)
    if not args.no_resnet:
        result["resnet18_fwd"] = resnet18_fwd(dev)
    if not args.no_small:
        result["small_workloads"] = small_configs(dev)
        result["weight_streaming"] = weight_streaming(dev)
        result["fused_update_quantize"] = fused_update(dev)
    from paper_1701_00485_amd import memory
    result["model_size"] = {k: {f: v[f] for f in ("params", "fp64_bytes", "tbn_bytes", "fp64_over_tbn")}
                            for k, v in memory.memory_table().items()}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
