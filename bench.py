#!/usr/bin/env python3
"""Benchmark of the PyraMiD-LSTM hot path on one MI355X; prints one JSON line.

Default run (the five workloads of the layer, seeded and synthetic; the MR
and EM shapes stand in for the MRBrainS13 and ISBI 2012 stacks of Section 3):
  value / ms_per_step  config 5: MR-like 48 x 240 x 240 x 3 volume, two
                       PyraMiD-LSTM layers (16, 32 hidden units, 3x3) each
                       followed by FC tanh (32, 64), linear + softmax over 4
                       classes, mean cross-entropy; forward + backward, fp32
                       (one timed step = one pass of the whole hot path)
  fwd                  config 2: the single-layer inference forward (six
                       sweeps + their sum) on the MR-like volume, fp32
  configs["3"]         config 3: EM-like 30 x 512 x 512 x 1 stack, one layer,
                       inference forward, fp32
  configs["4"]         config 4: 8 x 64^3 x 3, three layers (16, 32, 64) + FC
                       tanh + softmax, bf16 storage / fp32 accumulation, forward
  cpu_baseline         the fp64 oracle on the host cores (bounded samples)
Inputs are resident in HBM before timing.  Each figure carries the roofline
of its dominant kernel (algorithmic flops per launch / HIP-event launch time).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

Single workloads can be timed instead (--workload; not the headline):
    mr-layer      48 x 240 x 240 x 3, one layer (16) + FC tanh + softmax-CE,
                  fp32, forward + backward, with the config-2 forward
    stacked-bf16  config 4 alone          train-2layer  config 5 alone
    em-layer      config 3 alone
    image-2d      the 30 EM-like slices as a batch of 512 x 512 images through
                  one 2D layer (16 units, 3 taps), fp32, forward + backward
    paper-net     the network of the paper's experiments (7x7 filters,
                  16 / FC 25 / 32 / FC 45 / 64 -> output) on a 25 x 240 x 240 x 5
                  MR sub-volume, squared loss, fp32, forward + backward + update
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "voxel-direction LSTM updates/sec (fwd, fwd+bwd) + % peak MFMA, 1 MI355X"
UNIT = "voxel-direction updates/s"
PEAK_FP32_TFLOPS = 157.3     # MI355X dense fp32 MFMA
PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E


def phase_work(name, V, C, O, K=3):
    """(bound, algorithmic amount per pass, unit) of a library phase for one
    layer over V voxels.  Contraction flops count the dense K x K stencils."""
    G, KK = 4 * O, K * K
    if name.startswith("sweep_fwd"):
        return "mfma", 6 * V * 2 * KK * G * (C + O), "TFLOP/s"
    if name.startswith("sweep_bwd"):
        # recurrent transposed convolution (dh) plus the gate gradients
        return "mfma", 6 * V * 2 * KK * G * O, "TFLOP/s"
    if name.startswith("wgrad"):
        return "mfma", 6 * V * 2 * G * (KK * (C + O) + 1), "TFLOP/s"
    if name.startswith("dx"):
        return "mfma", 6 * V * 2 * KK * G * C, "TFLOP/s"
    if name.startswith("sum_dirs"):
        return "hbm", (6 + 1) * V * O * 4, "GB/s"
    if name.startswith("head_fused"):
        # reads h and the label, writes p (4 classes) and dL/dh per voxel
        return "hbm", V * (O * 4 + 4 + 4 * 4 + O * 4), "GB/s"
    if name.startswith("head_fwd"):
        # bf16 inference head: reads h, writes p (4 classes, fp32) per voxel
        return "hbm", V * (O * 2 + 4 * 4), "GB/s"
    return None, None, None


# Counter figures measured with rocprofv3 and committed under profiles/ as
# machine-readable lines (one per workload and bench phase):
#   traffic workload=W kernel=K mode=M bytes_per_pass=B src=S
#       HBM bytes (FETCH_SIZE + WRITE_SIZE, each calibrated against a copy of
#       known size) of the phase's kernels over one pass of the workload
#   mfma workload=W kernel=K flops_per_pass=F busy=U src=S
#       executed MFMA flops (SQ_INSTS_VALU_MFMA_MOPS_F32/BF16 x 512) and the
#       matrix units' busy fraction (SQ_VALU_MFMA_BUSY_CYCLES over
#       GRBM_GUI_ACTIVE x 128)
# S is the first 16 hex digits of the SHA-256 of the kernel's sources when
# measured (comments and whitespace aside); a figure whose sources changed
# since is reported as null.
PROFILES = os.path.join(ROOT, "profiles")
_STEP = ["sweep_step.hip", "common.h"]
KERNEL_SOURCES = {
    "sweep_fwd_mfma": ["sweep_fwd.hip", "strip_plan.h", "common.h", "coherent.h"],
    "sweep_bwd_mfma": ["sweep_bwd.hip", "strip_plan.h", "common.h", "coherent.h"],
    "wgrad_mfma": ["sweep_bwd.hip", "strip_plan.h", "common.h", "coherent.h"],
    "sweep_fwd_step": _STEP, "sweep_bwd_step": _STEP, "wgrad_step": _STEP, "dx_step": _STEP,
    "sweep_fwd_step_bf16": _STEP,
    "sum_dirs": ["generic.hip", "common.h"],
    "head_fused": ["fc.hip", "common.h"], "fc_tanh_fwd": ["fc.hip", "common.h"],
    "head_fwd": ["fc.hip", "common.h"],
    "fc_tanh_bwd": ["fc.hip", "common.h"], "softmax_ce": ["fc.hip", "common.h"],
}


def source_hash(kernel):
    """Hash of the code of the kernel's sources: comments and whitespace are
    dropped first, so that editing a comment keeps the measured figures."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_1506_07452_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


_PROFILE_LINES = None


def profile_lines():
    global _PROFILE_LINES
    if _PROFILE_LINES is None:
        _PROFILE_LINES = []
        if os.path.isdir(PROFILES):
            for fn in sorted(os.listdir(PROFILES)):
                if not fn.endswith(".md"):
                    continue
                for line in open(os.path.join(PROFILES, fn)):
                    if line.startswith(("traffic ", "mfma ")):
                        kind, rest = line.split(None, 1)
                        _PROFILE_LINES.append(
                            (kind, dict(kv.split("=", 1) for kv in rest.split())))
    return _PROFILE_LINES


def measured(kind, kernel, workload, mode=None):
    """The committed counter line for (kind, kernel, workload[, mode]), or
    None when there is none or the kernel's sources changed since."""
    if kernel not in KERNEL_SOURCES or workload is None:
        return None
    for k, f in profile_lines():
        if (k == kind and f.get("kernel") == kernel and f.get("workload") == workload and
                (mode is None or f.get("mode") == mode)):
            return f if f.get("src") == source_hash(kernel) else None
    return None


def counter_fields(name, workload, mode, passes, launches, algorithmic_per_pass):
    """traffic (HBM bytes per launch) and the MFMA figures of a phase from the
    committed profiles."""
    out = {"traffic": None, "mfma_executed_over_algorithmic": None, "mfma_busy": None}
    t = measured("traffic", name, workload, mode)
    if t is not None:
        out["traffic"] = int(float(t["bytes_per_pass"]) * passes / launches)
    m = measured("mfma", name, workload)
    if m is not None and algorithmic_per_pass:
        out["mfma_executed_over_algorithmic"] = round(
            float(m["flops_per_pass"]) / algorithmic_per_pass, 4)
        out["mfma_busy"] = round(float(m["busy"]), 4)
    return out


def roofline(phases, name, passes, V, C, O, mode="training", workload=None):
    ms, launches = phases[name]
    bound, amount, unit = phase_work(name, V, C, O)
    if bound is None:
        return None
    per_launch = amount * passes / launches
    avg_s = ms / 1e3 / launches
    if bound == "hbm":
        achieved, peak = per_launch / avg_s / 1e9, PEAK_HBM_GBS
    else:
        achieved, peak = per_launch / avg_s / 1e12, PEAK_FP32_TFLOPS
    out = {"kernel": name, "bound": bound, "achieved": round(achieved, 3), "peak": peak,
           "unit": unit, "frac": round(achieved / peak, 4)}
    out.update(counter_fields(name, workload, mode, passes, launches,
                              amount if bound == "mfma" else None))
    out.update({"launches_per_pass": launches // passes,
                "avg_launch_ms": round(ms / launches, 4)})
    return out


def layer_path(C, O, dtype, K=3):
    """Which forward kernels the library runs for a layer (inference with
    bf16 storage, training in fp32): the plane-step bf16 MFMA (bf16 storage,
    32 or 64 hidden units, or 16 with at most 8 input channels), the persistent
    sweeps (16 hidden units, at most 4 input channels, 3x3) or the plane-step
    fp32 MFMA; phase names end in _step_bf16, _mfma or _step."""
    if dtype == "bf16" and (O in (32, 64) or (O == 16 and C <= 8)):
        return "step_bf16"
    if O == 16 and C <= 4 and K == 3:
        return "mfma"
    return "step"


def dx_in_reverse(li, C, O, path):
    """Whether the library's staged reverse step computes dL/dx of this layer
    (layers after the first on the fp32 plane-step path with at most 32 units
    and 32 input channels, padded to 16); dx_step then only adds the
    directions."""
    return li > 0 and path == "step" and O <= 32 and (C + 15) // 16 * 16 <= 32


def network_roofline(phases, passes, V, shapes, dtype, K=3, workload=None, mode=None):
    """Roofline of the slowest phase of a multi-layer pass: its algorithmic
    work summed over the layers that ran it (the reverse step's includes
    dL/dx where it computes it)."""
    cand = {k: v for k, v in phases.items() if phase_work(k, 1, 1, 16)[0] == "mfma"}
    name = max(cand, key=lambda k: cand[k][0])
    ms, launches = phases[name]
    flops = 0
    for li, (C, O) in enumerate(shapes):
        path = layer_path(C, O, dtype, K)
        fused = dx_in_reverse(li, C, O, path)
        if name.startswith("dx"):
            if li > 0 and not fused:
                flops += phase_work(name, V, C, O, K)[1]
        elif name.endswith("_" + path):
            flops += phase_work(name, V, C, O, K)[1]
        if name == "sweep_bwd_step" and fused:
            flops += phase_work("dx", V, C, O, K)[1]
    achieved = flops * passes / (ms / 1e3) / 1e12
    peak = PEAK_BF16_TFLOPS if name.endswith("_bf16") else PEAK_FP32_TFLOPS
    out = {"kernel": name, "bound": "mfma", "achieved": round(achieved, 3),
           "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
    out.update(counter_fields(name, workload, mode, passes, launches, flops))
    out.update({"launches_per_pass": launches // passes,
                "avg_launch_ms": round(ms / launches, 4)})
    return out


def timed(step, args):
    """W untimed warm-up steps, then K steps bracketed by device
    synchronisation; per-phase HIP-event times of the K steps.  Raises if a
    persistent sweep reported a failed wait on the way."""
    import torch
    import paper_1506_07452_amd as P
    P.pyramid_lstm_device_status(clear=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    P.pyramid_lstm_timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / args.steps
    phases = P.pyramid_lstm_timing_read()
    P.pyramid_lstm_timing_enable(False)
    status = P.pyramid_lstm_device_status(clear=True)
    if status:
        raise RuntimeError("a persistent sweep's wait gave up during the run (status %d)"
                           % status)
    return t, phases


def phases_per_step(phases, steps):
    return {k: round(v[0] / steps, 4) for k, v in phases.items()}


def measure_network(args, cfg):
    """Config 4 (stacked, bf16 storage, forward), config 5 (two layers, fp32,
    training step) or the paper's network (cfg None), through the same entry
    points.  Returns (seconds per pass, phases, workload, config dict)."""
    import torch
    import synth
    from paper_1506_07452_amd.network import (LayerW, network_forward, network_train_step,
                                              workspace_for_layers)
    inst = synth.config(cfg) if cfg is not None else synth.make(synth.PAPER_NET)
    wl = inst.wl
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16

    def dev(a):
        return torch.from_numpy(a).to("cuda:0").to(tdt).contiguous()

    x = dev(inst.x)
    layers = [LayerW(dev(L.wx), dev(L.wh), dev(L.b)) for L in inst.layers]
    fcs = [(dev(w), dev(b)) for w, b in inst.fcs]
    head = (dev(inst.head[0]), dev(inst.head[1]))
    train = wl.labels
    labels = torch.from_numpy(inst.labels).to("cuda:0") if train else None
    ws = workspace_for_layers(x.shape, [(C, O, wl.K) for C, O in wl.layer_shapes()], tdt,
                              train, "cuda:0")
    torch.cuda.synchronize()

    # the paper's network trains with its own update (RMS-prop with momentum,
    # Section 3) inside the timed step
    opt = None
    if cfg is None:
        from paper_1506_07452_amd import RMSprop
        from paper_1506_07452_amd.network import network_gradients, network_parameters
        opt = RMSprop(network_parameters(layers, fcs, head))

    def step():
        if train:
            # the paper trains on the squared loss of Eq. (14)
            g = network_train_step(x, layers, fcs, head, labels, ws=ws,
                                   loss="sq" if cfg is None else "ce")
            if opt is not None:
                opt.step(network_gradients(g), 0)
            return g
        return network_forward(x, layers, fcs, head, ws=ws)

    t, phases = timed(step, args)
    conf = {"workload": wl.name + (" (squared loss)" if opt is not None else "") +
                        (", fwd+bwd" if train else ", fwd") +
                        (" + RMS-prop update" if opt is not None else ""),
            "N": wl.N, "D": wl.D, "H": wl.H, "W": wl.W, "C": wl.C, "hidden": wl.hidden,
            "fc": [wl.fc_width(i) for i in range(len(wl.hidden))], "K": wl.K,
            "storage": wl.dtype, "classes": wl.classes}
    del x, layers, fcs, head, labels, ws, step, opt
    torch.cuda.empty_cache()
    return t, phases, wl, conf


def network_summary(args, cfg):
    """A network workload as a JSON object: time, updates/s, contraction
    TFLOP/s and the roofline of its slowest phase."""
    t, phases, wl, conf = measure_network(args, cfg)
    train = wl.labels
    return {
        "config": conf, "ms_per_pass": round(t * 1e3, 4), "value": wl.vdu_per_pass() / t,
        "unit": UNIT, "dtype": wl.dtype,
        "tflops": None if train else round(wl.flops_per_pass() / t / 1e12, 3),
        "roofline": network_roofline(phases, args.steps, wl.voxels, wl.layer_shapes(),
                                     wl.dtype, wl.K, workload=None if cfg is None else
                                     "cfg%d" % cfg,
                                     mode="training" if train else "inference"),
        "phases_ms_per_step": phases_per_step(phases, args.steps),
    }


def layer_forward_summary(args, cfg):
    """Configs 2 and 3: one layer's inference forward (six sweeps and their
    sum), fp32.  Returns a JSON object with the forward sweep's roofline."""
    import torch
    import synth
    from paper_1506_07452_amd.network import LayerW, layer_forward, workspace_for
    inst = synth.config(cfg)
    wl = inst.wl
    x = torch.from_numpy(inst.x).to("cuda:0").contiguous()
    L = inst.layers[0]
    Ld = LayerW(*(torch.from_numpy(a).to("cuda:0").contiguous() for a in (L.wx, L.wh, L.b)))
    ws = workspace_for(x.shape, wl.hidden, False, torch.float32, False, "cuda:0")
    torch.cuda.synchronize()
    t, phases = timed(lambda: layer_forward(x, Ld, False, ws=ws), args)
    N, D, H, W, C = inst.x.shape
    O = wl.hidden[0]
    V = N * D * H * W
    flops = 6 * V * 2 * 9 * 4 * O * (C + O)
    name = next(k for k in phases if k.startswith("sweep_fwd"))
    roof = roofline(phases, name, args.steps, V, C, O, mode="inference",
                    workload="cfg%d" % cfg)
    del x, Ld, ws
    torch.cuda.empty_cache()
    return {"config": {"workload": wl.name, "N": N, "D": D, "H": H, "W": W, "C": C, "O": O},
            "ms_per_pass": round(t * 1e3, 4), "value": 6 * V / t, "unit": UNIT, "dtype": "f32",
            "tflops": round(flops / t / 1e12, 3),
            "frac_fp32_mfma_peak": round(flops / t / 1e12 / PEAK_FP32_TFLOPS, 4),
            "roofline": roof, "phases_ms_per_step": phases_per_step(phases, args.steps)}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_legs(threads_all):
    """The fp64 oracle, as it stands, on the host cores: bounded samples of
    the headline training step and of the config-2 forward (all threads), and
    single-thread forwards of configs 1-3 on bounded crops.  Each leg reports
    voxel-direction updates per second of what it ran."""
    import numpy as np
    import oracle
    import oracle.network as onet
    import synth

    legs = []

    def leg(cfg, crop, threads, what, fn, x):
        oracle.set_threads(threads)
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        nvox = int(np.prod(x.shape[:4]))
        layers = len(synth.CONFIGS[cfg].hidden)
        legs.append({"config": cfg, "what": what, "sample": "x".join(map(str, x.shape[1:4])) +
                     ("" if crop is None else " crop"), "threads": threads,
                     "seconds": round(dt, 2), "value": 6 * nvox * layers / dt})

    inst5 = synth.config(5)
    x5 = np.ascontiguousarray(inst5.x[:, :, :60, :60])
    lab5 = inst5.labels.reshape(inst5.x.shape[:4])[:, :, :60, :60].reshape(-1)
    lw5 = [(L.wx, L.wh, L.b) for L in inst5.layers]
    leg(5, (48, 60, 60), threads_all, "training step fwd+bwd (2 layers, FC, softmax-CE)",
        lambda: onet.backward(x5, lw5, inst5.fcs, inst5.head, lab5), x5)
    inst2 = synth.config(2)
    L2 = inst2.layers[0]
    leg(2, None, threads_all, "layer forward",
        lambda: oracle.forward(inst2.x, L2.wx, L2.wh, L2.b), inst2.x)
    inst1 = synth.config(1)
    L1 = inst1.layers[0]
    leg(1, None, 1, "layer forward", lambda: oracle.forward(inst1.x, L1.wx, L1.wh, L1.b),
        inst1.x)
    x2c = np.ascontiguousarray(inst2.x[:, :, :40, :40])
    leg(2, (48, 40, 40), 1, "layer forward", lambda: oracle.forward(x2c, L2.wx, L2.wh, L2.b),
        x2c)
    inst3 = synth.config(3)
    L3 = inst3.layers[0]
    x3c = np.ascontiguousarray(inst3.x[:, :, :56, :56])
    leg(3, (30, 56, 56), 1, "layer forward", lambda: oracle.forward(x3c, L3.wx, L3.wh, L3.b),
        x3c)
    oracle.set_threads(threads_all)
    head = legs[0]
    return {"value": head["value"], "unit": UNIT, "cores": head["threads"], "kind": "oracle",
            "sample": "oracle fp64 config-5 training step (2 layers fwd+bwd, FC tanh, "
                      "softmax-CE) on the 48x60x60 corner crop of the same volume, %.1f s on "
                      "%d threads" % (head["seconds"], head["threads"]),
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(), "legs": legs}


def bench_all(args):
    """The default run: config 5 as the headline, configs 2, 3, 4 beside it."""
    import torch
    torch.cuda.init()
    t5, phases5, wl5, conf5 = measure_network(args, 5)
    out = {
        "metric": METRIC, "value": wl5.vdu_per_pass() / t5, "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": t5 * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic", "config": conf5,
        "roofline": network_roofline(phases5, args.steps, wl5.voxels, wl5.layer_shapes(),
                                     wl5.dtype, wl5.K, workload="cfg5", mode="training"),
        "phases_ms_per_step": phases_per_step(phases5, args.steps),
    }
    out["fwd"] = layer_forward_summary(args, 2)
    out["configs"] = {"3": layer_forward_summary(args, 3), "4": network_summary(args, 4)}
    if not args.no_cpu_baseline:
        import oracle
        out["cpu_baseline"] = cpu_legs(oracle.threads())
    print(json.dumps(out), flush=True)


def bench_network(args, cfg):
    """One network workload as the whole JSON line."""
    s = network_summary(args, cfg)
    out = {"metric": METRIC, "value": s["value"], "unit": UNIT, "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": s["ms_per_pass"],
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": s["dtype"], "data": "synthetic", "config": s["config"],
           "tflops": s["tflops"], "roofline": s["roofline"],
           "phases_ms_per_step": s["phases_ms_per_step"]}
    print(json.dumps(out), flush=True)


def bench_em(args):
    """The EM-like stack (ISBI 2012 shape) through one layer, inference
    forward: six sweeps and their sum."""
    s = layer_forward_summary(args, 3)
    out = {"metric": METRIC, "value": s["value"], "unit": UNIT, "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": s["ms_per_pass"],
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic", "config": s["config"], "tflops": s["tflops"],
           "roofline": s["roofline"], "phases_ms_per_step": s["phases_ms_per_step"]}
    print(json.dumps(out), flush=True)


def bench_2d(args):
    """The 2D layer (four line sweeps, Section 2.1-2.2) over the EM-like
    slices as a batch of images: training forward + backward."""
    import torch
    import synth
    import paper_1506_07452_amd as P
    from paper_1506_07452_amd.network import LayerW, layer2d_backward, layer2d_forward
    N, H, W, C, O, K = 30, 512, 512, 1, 16, 3
    x, wx, wh, b = synth.image2d(N, H, W, C, O, K, seed=2048, scale=0.1)
    torch.cuda.init()
    dev = lambda a: torch.from_numpy(a).to("cuda:0").contiguous()
    xd, L = dev(x), LayerW(dev(wx), dev(wh), dev(b))
    s = P.shape2d_for(xd, O, K)
    ws = torch.empty(P.pyramid_lstm2d_workspace_size(s, 1), dtype=torch.uint8, device="cuda:0")
    dh = torch.ones((N, H, W, O), device="cuda:0")

    def step():
        h, saved = layer2d_forward(xd, L, training=True, ws=ws)
        return layer2d_backward(xd, L, saved, dh, ws=ws)

    t, phases = timed(step, args)
    V = N * H * W
    # algorithmic flops per pixel-direction: forward 2 K 4O (C + O); reverse
    # 2 K 4O O; weight gradients 2 4O (K (C + O) + 1); dL/dx 2 K 4O C
    G = 4 * O
    work = {"sweep_fwd_step": 2 * K * G * (C + O), "sweep_bwd_step": 2 * K * G * O,
            "wgrad_step": 2 * G * (K * (C + O) + 1), "dx_step": 2 * K * G * C}
    name = max((k for k in phases if k in work), key=lambda k: phases[k][0])
    ms, launches = phases[name]
    per_launch = 4 * V * work[name] * args.steps / launches
    achieved = per_launch / (ms / 1e3 / launches) / 1e12
    out = {
        "metric": METRIC, "value": 4 * V / t, "unit": UNIT, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "2D PyraMiD-LSTM, 30 EM-like 512x512 slices as images, O=16, "
                               "1x3 filters, fwd+bwd", "N": N, "H": H, "W": W, "C": C, "O": O,
                   "K": K},
        "roofline": {"kernel": name, "bound": "mfma", "achieved": round(achieved, 3),
                     "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_FP32_TFLOPS, 4), "traffic": None,
                     "launches_per_pass": launches // args.steps,
                     "avg_launch_ms": round(ms / launches, 4)},
        "phases_ms_per_step": {k: round(v[0] / args.steps, 4) for k, v in phases.items()},
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_step(inst_cfg, crop):
    """The fp64 oracle (as is) on a bounded crop of the single-layer step."""
    import numpy as np
    import oracle
    import oracle.network as onet
    D, H, W = crop
    x = inst_cfg.x[:, :D, :H, :W, :]
    lab = inst_cfg.labels.reshape(inst_cfg.x.shape[:4])[:, :D, :H, :W].reshape(-1)
    layers = [(L.wx, L.wh, L.b) for L in inst_cfg.layers]
    t0 = time.perf_counter()
    onet.backward(x, layers, inst_cfg.fcs, inst_cfg.head, lab)
    dt = time.perf_counter() - t0
    vdu = 6 * int(np.prod(x.shape[:4]))
    return {"value": vdu / dt, "unit": UNIT, "cores": oracle.threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": "oracle fp64 training step (layer fwd+bwd, FC tanh, softmax-CE) on a "
                      "%dx%dx%dx%d crop of the same volume, %.1f s" % (D, H, W, x.shape[-1], dt)}


def bench_mr_layer(args):
    """48 x 240 x 240 x 3, one layer (16) + FC tanh 32 + softmax-CE, fp32,
    forward + backward, with the config-2 inference forward beside it."""
    import torch
    import synth
    from paper_1506_07452_amd.network import LayerW, network_train_step, workspace_for

    def dev(a):
        return torch.from_numpy(a).to("cuda:0").contiguous()

    wl = synth.Workload("MR-like 48x240x240x3 O=16 step", 1, 48, 240, 240, 3, [16], fc=True,
                        classes=4, labels=True, kind="mr", cfg=2)
    inst = synth.make(wl)
    N, D, H, W, C = inst.x.shape
    O = wl.hidden[0]
    V = N * D * H * W
    torch.cuda.init()
    x = dev(inst.x)
    layers = [LayerW(dev(L.wx), dev(L.wh), dev(L.b)) for L in inst.layers]
    fcs = [(dev(w), dev(b)) for w, b in inst.fcs]
    head = (dev(inst.head[0]), dev(inst.head[1]))
    labels = torch.from_numpy(inst.labels).to("cuda:0")
    ws = workspace_for(x.shape, wl.hidden, True, torch.float32, True, "cuda:0")
    torch.cuda.synchronize()

    def step():
        return network_train_step(x, layers, fcs, head, labels, ws=ws,
                                  fused_head=not args.separate_head)

    t_step, phases = timed(step, args)
    del x, layers, fcs, head, labels, ws
    torch.cuda.empty_cache()
    dom = max(phases, key=lambda k: phases[k][0])
    out = {
        "metric": METRIC, "value": 6 * V / t_step, "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": t_step * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "MR-like 48x240x240x3 volume, one PyraMiD-LSTM layer (O=16, "
                               "3x3, 6 directions) + FC tanh 32 + softmax-CE head, fwd+bwd",
                   "N": N, "D": D, "H": H, "W": W, "C": C, "O": O, "classes": 4},
        "fwd": layer_forward_summary(args, 2),
        # the first layer of the 2-layer step is this layer (same kernels and
        # shapes): its counter figures apply
        "roofline": roofline(phases, dom, args.steps, V, C, O,
                             workload="cfg5" if dom in ("sweep_fwd_mfma", "sweep_bwd_mfma",
                                                        "wgrad_mfma") else None),
        "phases_ms_per_step": phases_per_step(phases, args.steps),
    }
    if not args.no_cpu_baseline:
        crop = tuple(int(v) for v in args.cpu_crop.split("x"))
        out["cpu_baseline"] = cpu_baseline_step(inst, crop)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-crop", default="48x120x120",
                    help="crop of the mr-layer workload's CPU baseline")
    ap.add_argument("--separate-head", action="store_true",
                    help="mr-layer: run the FC / softmax head as separate kernels")
    ap.add_argument("--workload", default="all",
                    choices=["all", "mr-layer", "em-layer", "image-2d", "stacked-bf16",
                             "train-2layer", "paper-net"],
                    help="all: config 5 as the headline with configs 2-4 beside it (default)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 1 GiB device-to-device three times (a plain copy kernel "
                         "of known size, to scale rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the six sweeps of a layer run concurrently "
              "on a single MI355X and the library has no multi-GPU path (--gpus 1).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
    if args.workload == "all":
        bench_all(args)
    elif args.workload == "mr-layer":
        bench_mr_layer(args)
    elif args.workload == "em-layer":
        bench_em(args)
    elif args.workload == "image-2d":
        bench_2d(args)
    else:
        bench_network(args, {"stacked-bf16": 4, "train-2layer": 5, "paper-net": None}[
            args.workload])
    release_device()


def copy_calibration():
    """Three device-to-device copies of 1 GiB: a plain copy kernel of known
    size that scales rocprofv3's FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    src = torch.zeros(1 << 28, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def release_device():
    """Leave nothing of ours on the device at interpreter exit: timing off
    (its events destroyed), the stream drained, torch's cached blocks
    returned to the runtime."""
    import gc
    import torch
    import paper_1506_07452_amd as P
    P.pyramid_lstm_timing_enable(False)
    torch.cuda.synchronize()
    gc.collect()
    torch.cuda.empty_cache()
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
