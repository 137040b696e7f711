#!/usr/bin/env python3
"""Benchmark of the selective-differentiation layers on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Headline step: the bf16 Linear stack X[4096,1024] -> 1024->4096->1024->4096->1024
with every weight frozen and biases trainable (mask = input + bias per layer):
four forward GEMMs, then four input-gradient GEMMs and four bias-gradient
reductions, all through the C ABI of libmemsave.so.  `value` is the
algorithmic TFLOP/s of the launched contractions (forward + input gradient;
the weight-gradient GEMMs are skipped by the mask) with every input resident
in HBM.  The line also carries the ledger's retained activation bytes under
the selective mask and under an all-true mask, the roofline of the dominant
kernel, the other synthetic workloads as context, and the CPU oracle timed on
a bounded sample.  The K timed steps carry no per-launch instrumentation; the
roofline's kernel time comes from a second pass over K steps in which the
library brackets every GEMM launch with HIP events on its stream.

One JSON line goes to stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "conv/linear fwd+bwd TFLOP/s (frozen W) + saved-activation bytes vs full AD"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 (matrix and vector)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ FLOP / byte accounting
def layer_flops(spec, mask: int) -> dict:
    """Algorithmic FLOP (2 x multiply-adds) of the contractions a layer
    launches: forward always, input gradient iff INPUT, weight gradient iff
    WEIGHT.  BN, pooling and bias work is not counted."""
    if spec.kind == "conv2d":
        n, c, _, _ = spec.in_shape
        _, k, p, q = spec.out_shape()
        r, s = spec.ksize
        f = 2 * n * p * q * k * c * r * s
    elif spec.kind == "conv_transpose2d":
        # the convolution it is the adjoint of: every input pixel meets every
        # tap and every (C_in, C_out) pair
        n, ci, h, w = spec.in_shape
        r, s = spec.ksize
        f = 2 * n * h * w * ci * spec.out_ch * r * s
    elif spec.kind == "linear":
        m, kin = spec.in_shape
        f = 2 * m * kin * spec.out_ch
    else:
        return {"fwd": 0, "dgrad": 0, "wgrad": 0}
    return {"fwd": f, "dgrad": f if mask & 1 else 0, "wgrad": f if mask & 2 else 0}


def numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


# ------------------------------------------------------------------ timing helpers
def time_chains(chains, steps, warmup, backward=True):
    import torch
    for _ in range(warmup):
        for c in chains:
            c.forward()
        if backward:
            for c in chains:
                c.backward()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        for c in chains:
            c.forward()
        if backward:
            for c in chains:
                c.backward()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def ledger_peak_of_forward(chains):
    """Peak retained activation bytes over one forward of `chains`."""
    import torch
    import paper_2404_12406_amd as ms
    torch.cuda.synchronize()
    live0, _ = ms.ledger_read()
    ms.ledger_reset()
    for c in chains:
        c.forward()
    torch.cuda.synchronize()
    _, peak = ms.ledger_read()
    return peak - live0


def with_masks(w, fn):
    """A copy of workload w with every layer's mask replaced by fn(layer)."""
    import copy
    w2 = copy.deepcopy(w)
    for l in w2.layers:
        l.mask = fn(l)
    return w2


def all_true(l):
    if l.kind == "avgpool":
        return 1
    return 1 | 2 | (4 if l.has_bias else 0)


# ------------------------------------------------------------------ recorded counters
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_linear_stack_bf16_hbm_counters.md")
GEMM_SOURCES = ("paper_2404_12406_amd/csrc/kernels/gemm_bf16.hip", "paper_2404_12406_amd/csrc/kernels/common.h")


def recorded_traffic(key: str):
    """HBM bytes per launch of the forward ("fwd") or input-gradient
    ("dgrad") GEMM from the committed FETCH_SIZE / WRITE_SIZE counter
    summary, or None when the GEMM sources changed since the counters were
    taken (or the summary is absent)."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    field = f"traffic_bytes_per_launch_{key}: "
    fields = dict(l.split(": ", 1) for l in text.splitlines() if l.startswith((field, "kernel_sources_sha256: ")))
    h = hashlib.sha256()
    for p in GEMM_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    if fields.get("kernel_sources_sha256", "").strip() != h.hexdigest() or field[:-2] not in fields:
        return None
    return int(fields[field[:-2]])


# ------------------------------------------------------------------ headline
def headline(steps, warmup):
    import torch
    import paper_2404_12406_amd as ms
    from synth import draw, gpu
    from synth import workloads as wl

    w = wl.linear_stack_bf16()
    ca = draw.chains(w)[0]
    chain = gpu.build_chain(ca, "bf16")
    fl = [layer_flops(l, l.mask) for l in w.layers]
    flop_step = sum(f["fwd"] + f["dgrad"] + f["wgrad"] for f in fl)
    log(f"[bench] headline {w.name}: {flop_step / 1e9:.2f} GFLOP per step; warmup {warmup}")
    for _ in range(warmup):
        chain.forward()
        chain.backward()
    torch.cuda.synchronize()
    # Pass 1, the headline: K steps timed with one event pair on the stream,
    # nothing else recorded.
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record()
    for _ in range(steps):
        chain.forward()
        chain.backward()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / steps
    # Pass 2, the roofline: the same K steps again with the library
    # bracketing each forward / input-gradient GEMM launch with HIP events on
    # the stream it launches on.  The event pairs cost a few microseconds per
    # launch, which is why they stay out of pass 1.  The dominant kernel is
    # the mode with the larger summed GPU time.
    ms.profile_start(ms.PROF_FWD | ms.PROF_DGRAD)
    t0.record()
    for _ in range(steps):
        chain.forward()
        chain.backward()
    t1.record()
    torch.cuda.synchronize()
    ms_step_profiled = t0.elapsed_time(t1) / steps
    kern = {}
    for name, kind, key in (("forward", ms.PROF_FWD, "fwd"), ("input-gradient", ms.PROF_DGRAD, "dgrad")):
        n, tot = ms.profile_read(kind)
        flop = sum(f[key] for f in fl) * steps
        kern[key] = {"name": name, "key": key, "launches": n, "ms": tot, "flop": flop}
    ms.profile_start(0)
    dom = max(kern.values(), key=lambda k: k["ms"])
    assert dom["launches"] == steps * len(w.layers), dom
    avg_ms = dom["ms"] / dom["launches"]
    achieved = dom["flop"] / (dom["ms"] * 1e-3) / 1e12
    value = flop_step / (ms_step * 1e-3) / 1e12
    for k in kern.values():
        log(f"[bench]   {k['name']} GEMM: {k['launches']} launches, avg {k['ms'] / max(k['launches'], 1) * 1e3:.1f} us, "
            f"{k['flop'] / max(k['ms'], 1e-9) / 1e9:.1f} TFLOP/s")
    log(f"[bench] headline {ms_step:.3f} ms/step, {value:.1f} TFLOP/s (host wall {wall * 1e3 / steps:.3f} ms/step); "
        f"profiled pass {ms_step_profiled:.3f} ms/step, dominant {dom['name']} GEMM = {achieved:.1f} TFLOP/s")

    sel = ledger_peak_of_forward([chain])
    chain.backward()
    wt = with_masks(w, all_true)
    full = gpu.build_chain(draw.chains(wt)[0], "bf16")
    allb = ledger_peak_of_forward([full])
    full.backward()
    torch.cuda.synchronize()
    del full
    return {
        "workload": w,
        "ms_per_step": ms_step,
        "value": value,
        "flop_step": flop_step,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic(dom["key"]),
                     "kernel": f"ms::g2::gemm_kernel ({dom['name']} GEMM of the Linear layers)",
                     "flop_per_launch": dom["flop"] // dom["launches"], "avg_launch_us": round(avg_ms * 1e3, 2),
                     "launches": dom["launches"], "pass_ms_per_step": round(ms_step_profiled, 4),
                     # the input-gradient launches also take the layer's bias
                     # gradient along: each block adds its share of dy's
                     # columns (dy read a second time) after the contraction
                     "fused": ("bias-gradient column sums of dy (8 or 32 MiB re-read per launch, no FLOP counted)"
                               if dom["key"] == "dgrad" else None)},
        "saved": {"selective": sel, "all_true": allb},
    }


# ------------------------------------------------------------------ context workloads
def run_workload(w, steps, warmup, backward=True):
    import torch
    from synth import draw, gpu
    chains = gpu.build_chains(draw.chains(w), w.dtype)
    fl = [layer_flops(l, l.mask) for l in w.layers]
    flop = sum(f["fwd"] + (f["dgrad"] + f["wgrad"] if backward else 0) for f in fl)
    ms_step = time_chains(chains, steps, warmup, backward)
    sel = ledger_peak_of_forward(chains)
    if backward:
        for c in chains:
            c.backward()
    torch.cuda.synchronize()
    tflops = flop / (ms_step * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
    out = {"ms_per_step": round(ms_step, 4), "gflop": round(flop / 1e9, 3), "tflops": round(tflops, 2),
           "frac_of_peak": round(tflops / peak, 4), "saved_selective": sel}
    del chains
    torch.cuda.empty_cache()
    return out


def bn_bandwidth(steps, warmup):
    """BN-eval forward of the ResNet-18-shaped stack's 17 BN layers, each on
    its own seeded input; HBM bytes = read x + write y.

    * per layer: the last-level cache is evicted by a 512 MiB read sweep (a
      write sweep would leave dirty lines whose write-back competes with the
      timed kernel), then one launch is timed by the library's HIP events
      around it (this includes the launch's dispatch latency, a few us);
    * stack: the 17 launches back to back, `steps` times, between two events
      (inputs and outputs together exceed the cache, so every pass streams
      from HBM)."""
    import torch
    import paper_2404_12406_amd as ms
    import synth
    from synth import draw, gpu
    from synth import workloads as wl
    w = wl.resnet18_shaped_bf16()
    big = torch.ones(1 << 27, dtype=torch.float32, device="cuda")
    layers = []
    for i, l in enumerate(w.layers):
        if l.kind != "bn_eval":
            continue
        la = draw.layer_arrays(l, "bf16")
        x = gpu.dev(synth.normal(l.in_shape, 3900 + i, dtype="bf16"), "bf16")
        spec = ms.BatchNormEval(gpu.dev(la.running_mean, "bf16"), gpu.dev(la.running_var, "bf16"), l.eps)
        p = ms.PreparedLayer(spec, x, gpu.dev(la.W, "bf16"), gpu.dev(la.b, "bf16"), 0)
        layers.append((l, p, 2 * numel(l.in_shape) * 2))
    for _ in range(warmup):
        for _, p, _ in layers:
            p.forward()
    torch.cuda.synchronize()
    res = []
    for l, p, nbytes in layers:
        ms.profile_start(ms.PROF_BN)
        for _ in range(steps):
            big.sum()
            p.forward()
        torch.cuda.synchronize()
        n, tot = ms.profile_read(ms.PROF_BN)
        ms.profile_start(0)
        assert n == steps, (n, steps)
        t = tot / n
        res.append({"layer": l.name, "bytes": nbytes, "us": round(t * 1e3, 2),
                    "GBs": round(nbytes / (t * 1e-3) / 1e9, 1)})
    del big
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        for _, p, _ in layers:
            p.forward()
    e1.record()
    torch.cuda.synchronize()
    st = e0.elapsed_time(e1) / steps
    tot_b = sum(b for _, _, b in layers)
    best = max(res, key=lambda r: r["bytes"])
    return {"layers": res,
            "largest_layer": {"layer": best["layer"], "GBs": best["GBs"],
                              "frac_of_hbm": round(best["GBs"] / PEAK_HBM_GBS, 4)},
            "stack": {"bytes": tot_b, "us": round(st * 1e3, 2), "GBs": round(tot_b / (st * 1e-3) / 1e9, 1),
                      "frac_of_hbm": round(tot_b / (st * 1e-3) / 1e9 / PEAK_HBM_GBS, 4), "launches": len(layers)}}


def relu_bandwidth(steps, warmup):
    """ReLU with a 1-bit saved mask (Sec. 2.2.2) on the stem-output tensor of
    the ResNet-18-shaped stack (64 x 64 x 112 x 112 bf16, channels-last).

    HBM bytes per launch: forward reads x and writes y and the mask
    (2 * 2 * n + n / 8), backward reads dy and the mask and writes dx (the
    same).  Each launch is timed by the library's HIP events after a 512 MiB
    read sweep evicts the cache.  Retained bytes: this library's mask, the
    paper's one-byte boolean mask, stock PyTorch's saved output."""
    import torch
    import paper_2404_12406_amd as ms
    shape = (64, 64, 112, 112)
    n = 64 * 64 * 112 * 112
    g = torch.Generator(device="cuda").manual_seed(4242)
    x = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    gy = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    gx = torch.empty_like(x)
    p = ms.PreparedLayer(ms.ReLU(), x, mask=ms.MASK_INPUT, grad_y=gy, grad_x=gx)
    big = torch.ones(1 << 27, dtype=torch.float32, device="cuda")
    for _ in range(max(1, warmup)):
        p.forward()
        p.backward()
    torch.cuda.synchronize()
    nbytes = 2 * 2 * n + n // 8
    out = {"shape": list(shape), "dtype": "bf16", "bytes_per_launch": nbytes}
    # forwards alone (a prepared layer frees its previous record itself), then
    # forward + backward pairs: the backward time is the difference of the
    # summed event times
    ms.profile_start(ms.PROF_ACT)
    for _ in range(steps):
        big.sum()
        p.forward()
    torch.cuda.synchronize()
    cnt, t_fwd = ms.profile_read(ms.PROF_ACT)
    assert cnt == steps, (cnt, steps)
    ms.profile_start(ms.PROF_ACT)
    for _ in range(steps):
        big.sum()
        p.forward()
        big.sum()
        p.backward()
    torch.cuda.synchronize()
    cnt, t_both = ms.profile_read(ms.PROF_ACT)
    ms.profile_start(0)
    assert cnt == 2 * steps, (cnt, steps)
    for name, ms_tot in (("forward", t_fwd), ("backward", t_both - t_fwd)):
        us = ms_tot / steps * 1e3
        out[name] = {"us": round(us, 2), "GBs": round(nbytes / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    out["saved_bytes"] = {"bits": ms.relu_mask_bytes(n), "one_byte_bool": n, "stock_output": 2 * n}
    del big
    return out


def dropout_bandwidth(steps, warmup):
    """Dropout that draws its mask again in backward (Sec. 2.2.2) on the
    stem-output tensor of the ResNet-18-shaped stack (64 x 64 x 112 x 112
    bf16, channels-last) and on the FFN hidden activation of the encoder
    (8192 x 3072 bf16), p = 0.1.

    HBM bytes per launch: read the input, write the output (2 * 2 * n); no
    mask is read or written.  ALU work per launch: one Philox4x32-10 block
    per 4 elements.  Each launch is timed by the library's HIP events after a
    512 MiB read sweep evicts the cache.  Retained bytes: this library keeps
    the generator state (0 bytes), stock PyTorch a one-byte mask (n)."""
    import torch
    import paper_2404_12406_amd as ms
    big = torch.ones(1 << 27, dtype=torch.float32, device="cuda")
    out = {}
    for name, shape in (("stem_output", (64, 64, 112, 112)), ("ffn_hidden", (8192, 3072))):
        n = numel(shape)
        g = torch.Generator(device="cuda").manual_seed(4343)
        x = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16)
        if len(shape) == 4:
            x = x.contiguous(memory_format=torch.channels_last)
        gy = torch.randn_like(x)
        gx = torch.empty_like(x)
        p = ms.PreparedLayer(ms.Dropout(0.1, 0x5EED, 0), x, mask=ms.MASK_INPUT, grad_y=gy, grad_x=gx)
        for _ in range(max(1, warmup)):
            p.forward()
            p.backward()
        torch.cuda.synchronize()
        nbytes = 2 * 2 * n
        res = {"shape": list(shape), "dtype": "bf16", "p": 0.1, "bytes_per_launch": nbytes,
               "philox_blocks_per_launch": ms.dropout_blocks(n)}
        ms.profile_start(ms.PROF_ACT)
        for _ in range(steps):
            big.sum()
            p.forward()
        torch.cuda.synchronize()
        cnt, t_fwd = ms.profile_read(ms.PROF_ACT)
        assert cnt == steps, (cnt, steps)
        ms.profile_start(ms.PROF_ACT)
        for _ in range(steps):
            big.sum()
            p.forward()
            big.sum()
            p.backward()
        torch.cuda.synchronize()
        cnt, t_both = ms.profile_read(ms.PROF_ACT)
        ms.profile_start(0)
        assert cnt == 2 * steps, (cnt, steps)
        for pas, ms_tot in (("forward", t_fwd), ("backward", t_both - t_fwd)):
            us = ms_tot / steps * 1e3
            res[pas] = {"us": round(us, 2), "GBs": round(nbytes / (us * 1e-6) / 1e9, 1),
                        "frac_of_hbm": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                        "G_elements_per_s": round(n / (us * 1e-6) / 1e9, 1)}
        res["saved_bytes"] = {"generator_state": 0, "stock_one_byte_mask": n}
        out[name] = res
        del p, x, gy, gx
    del big
    torch.cuda.empty_cache()
    return out


def conv3d_throughput(steps, warmup):
    """One training step (forward, input and weight gradients, bias
    gradient) of a bf16 Conv3d 64 -> 64, 3x3x3, pad 1 on
    x = (8, 64, 16, 56, 56), and of a bf16 ConvTranspose3d 128 -> 64,
    2x2x2, stride 2 on x = (8, 128, 8, 28, 28) (the 3-D layers run as the
    2-D GEMMs on depth-folded inputs).  FLOP: 3 x 2 N Do P Q K C T R S."""
    import torch
    import paper_2404_12406_amd as ms
    out = {}
    cases = (("conv3d_64x64_3x3x3", ms.Conv3d(1, 1), (8, 64, 16, 56, 56), (64, 64, 3, 3, 3)),
             ("conv_transpose3d_128x64_2x2x2_s2", ms.ConvTranspose3d(2, 0), (8, 128, 8, 28, 28), (128, 64, 2, 2, 2)))
    for name, spec, xs, ws in cases:
        g = torch.Generator(device="cuda").manual_seed(4545)
        cl = torch.channels_last_3d
        x = torch.randn(xs, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=cl)
        w = (0.05 * torch.randn(ws, generator=g, device="cuda")).to(torch.bfloat16).contiguous(memory_format=cl)
        cy = ws[1] if isinstance(spec, ms.ConvTranspose3d) else ws[0]
        b = torch.zeros(cy, device="cuda", dtype=torch.bfloat16)
        yshape = ms.output_shape(spec, x, w)
        gy = torch.randn(yshape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=cl)
        p = ms.PreparedLayer(spec, x, w, b, mask=7, grad_y=gy, grad_x=torch.empty_like(x),
                             grad_W=torch.empty_like(w), grad_b=torch.empty_like(b))
        if isinstance(spec, ms.ConvTranspose3d):
            f = 2 * numel(xs) * ws[1] * ws[2] * ws[3] * ws[4]
        else:
            f = 2 * numel(yshape) * ws[1] * ws[2] * ws[3] * ws[4]
        for _ in range(max(1, warmup)):
            p.forward()
            p.backward()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            p.forward()
            p.backward()
        e1.record()
        torch.cuda.synchronize()
        step_ms = e0.elapsed_time(e1) / steps
        tf = 3 * f / (step_ms * 1e-3) / 1e12
        out[name] = {"x": list(xs), "W": list(ws), "ms_per_step": round(step_ms, 4), "gflop": round(3 * f / 1e9, 2),
                     "tflops": round(tf, 1), "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4)}
        del p, x, w, gy
    torch.cuda.empty_cache()
    return out


PROBE_SHAPES = {"conv2d": (256, 8, 256, 256), "conv_transpose2d": (256, 8, 256, 256),
                "conv1d": (4096, 8, 4096), "conv_transpose1d": (4096, 8, 4096),
                "conv3d": (64, 8, 64, 64, 64), "conv_transpose3d": (64, 8, 64, 64, 64)}


def memory_probe(kind: str = "conv2d", depth: int = 16):
    """The synthetic deep CNN of Sec. 2.1 (Fig. 1) at the paper's shape, and
    its App. B repetitions with the other layers linear in input and weight:
    `depth` bias-free size-preserving layers with 8 channels and kernel 3
    (conv2d / conv_transpose2d on (256, 8, 256, 256), conv1d /
    conv_transpose1d on (4096, 8, 4096), conv3d / conv_transpose3d on
    (64, 8, 64, 64, 64); fp32, 512 MiB per layer input), in
    three cases -- every layer and the input differentiable, layers 4+
    differentiable, only layer 4 differentiable -- built from torch.nn and
    converted to the library's layers, and the same model with stock PyTorch
    layers for context.  Reported: bytes the allocator holds after the
    forward pass (beyond the input and the output) and its forward peak, in
    MiB."""
    import torch
    from torch import nn
    from paper_2404_12406_amd import autograd as msa
    xs = PROBE_SHAPES[kind]
    per_input = numel(xs) * 4
    make = {"conv2d": lambda: nn.Conv2d(8, 8, 3, padding=1, bias=False),
            "conv_transpose2d": lambda: nn.ConvTranspose2d(8, 8, 3, padding=1, bias=False),
            "conv1d": lambda: nn.Conv1d(8, 8, 3, padding=1, bias=False),
            "conv_transpose1d": lambda: nn.ConvTranspose1d(8, 8, 3, padding=1, bias=False),
            "conv3d": lambda: nn.Conv3d(8, 8, 3, padding=1, bias=False),
            "conv_transpose3d": lambda: nn.ConvTranspose3d(8, 8, 3, padding=1, bias=False)}[kind]
    out = {"layer": kind, "shape": list(xs), "depth": depth, "dtype": "f32", "layer_input_MiB": per_input / 2 ** 20}
    for impl in ("library", "stock_pytorch"):
        res = {}
        for case in ("all", "layers_4_plus", "layer_4_only"):
            torch.manual_seed(0)
            convs = [make().cuda() for _ in range(depth)]
            for i, c in enumerate(convs):
                layer = i + 1
                c.weight.requires_grad_(case == "all" or (case == "layers_4_plus" and layer >= 4)
                                        or (case == "layer_4_only" and layer == 4))
                if impl == "stock_pytorch" and len(xs) >= 4:
                    c.weight.data = c.weight.data.contiguous(
                        memory_format=torch.channels_last if len(xs) == 4 else torch.channels_last_3d)
            net = nn.Sequential(*convs)
            if impl == "library":
                msa.convert(net)
            x = torch.randn(xs, device="cuda")
            if len(xs) == 4:
                x = x.contiguous(memory_format=torch.channels_last)
            elif len(xs) == 5:
                x = x.contiguous(memory_format=torch.channels_last_3d)
            else:
                x = x.transpose(1, 2).contiguous().transpose(1, 2)
            x.requires_grad_(case == "all")
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            y = net(x)
            torch.cuda.synchronize()
            held = torch.cuda.memory_allocated() - base - y.numel() * y.element_size()
            peak = torch.cuda.max_memory_allocated() - base
            res[case] = {"held_MiB": round(held / 2 ** 20, 1), "held_layer_inputs": round(held / per_input, 3),
                         "peak_MiB": round(peak / 2 ** 20, 1)}
            del y, net, convs, x
            torch.cuda.empty_cache()
        out[impl] = res
    return out


def extras(steps, warmup):
    from synth import workloads as wl
    out = {}
    steps = max(3, min(steps, 10))
    warmup = max(1, min(warmup, 3))
    jobs = [("single_conv2d_f32", wl.single_conv_f32(), True),
            ("resnet18_shaped_bf16", wl.resnet18_shaped_bf16(), True),
            ("resnet18_shaped_bf16_input", wl.resnet18_shaped_bf16(input_requires_grad=True), True),
            ("encoder_linears_bf16", wl.encoder_linears_bf16(), True),
            ("decoder_convt_bf16", wl.decoder_convt_bf16(), True)]
    for mk in ("00", "10", "01", "11"):
        jobs.append((f"conv_sweep_3x3_{mk}", wl.conv_sweep_bf16(mk), True))
        jobs.append((f"conv_sweep_1x1_{mk}", wl.conv_sweep_bf16(mk, pointwise=True), True))
    for name, w, bwd in jobs:
        t0 = time.time()
        out[name] = run_workload(w, steps, warmup, bwd)
        log(f"[bench] {name}: {out[name]} ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["bn_eval_forward_resnet18_shaped"] = bn = bn_bandwidth(steps, warmup)
    log(f"[bench] bn: stack {bn['stack']['GBs']} GB/s, largest layer {bn['largest_layer']} ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["fig1_synthetic_cnn_memory"] = f1 = memory_probe("conv2d")
    log(f"[bench] fig1 probe: library {f1['library']}, stock {f1['stock_pytorch']} ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["conv3d_training_step_bf16"] = c3 = conv3d_throughput(steps, warmup)
    log(f"[bench] 3-D convolutions: {c3} ({time.time() - t0:.1f}s)")
    out["appB_layer_memory"] = {}
    for kind in ("conv_transpose2d", "conv1d", "conv_transpose1d", "conv3d", "conv_transpose3d"):
        t0 = time.time()
        out["appB_layer_memory"][kind] = pr = memory_probe(kind)
        log(f"[bench] App. B probe {kind}: library {pr['library']}, stock {pr['stock_pytorch']} "
            f"({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["dropout_regenerated_mask"] = dr = dropout_bandwidth(steps, warmup)
    log(f"[bench] dropout: " + ", ".join(f"{k} fwd {v['forward']} bwd {v['backward']}" for k, v in dr.items())
        + f" ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["relu_bitmask_stem_output"] = rl = relu_bandwidth(steps, warmup)
    log(f"[bench] relu: forward {rl['forward']}, backward {rl['backward']}, saved {rl['saved_bytes']} "
        f"({time.time() - t0:.1f}s)")
    return out


# ------------------------------------------------------------------ CPU baseline
def cpu_baseline(target_s: float = 20.0):
    """The oracle (fp64 C loops, OpenMP) on the first `rows` rows of the
    headline workload: forward, input gradient and bias gradient of the four
    layers; the rate scales to the whole step by its FLOP count."""
    import numpy as np
    import oracle
    from synth import draw
    from synth import workloads as wl
    w = wl.linear_stack_bf16()
    ca = draw.chains(w)[0]

    def run(rows):
        x = ca.x[:rows]
        acts = [x]
        t = time.perf_counter()
        for la in ca.layers:
            acts.append(oracle.round_to(oracle.linear_forward(acts[-1], la.W, la.b), "bf16"))
        g = ca.grad_y[:rows]
        for i in range(len(ca.layers) - 1, -1, -1):
            oracle.linear_bias_grad(g)
            g = oracle.round_to(oracle.linear_input_grad(g, ca.layers[i].W), "bf16")
        return time.perf_counter() - t

    per_row = sum(2 * 2 * l.in_shape[1] * l.out_ch for l in w.layers)   # fwd + dgrad
    t = run(8)
    rows = int(min(ca.x.shape[0], max(8, 8 * target_s / max(t, 1e-3))))
    t = run(rows)
    tflops = rows * per_row / t / 1e12
    return {"value": round(tflops, 6), "unit": "TFLOP/s", "cores": oracle.threads(), "kind": "oracle",
            "sample": f"first {rows} of 4096 rows of the Linear stack, forward + input grad + bias grad "
                      f"of all 4 layers ({rows * per_row / 1e9:.2f} GFLOP in {t:.1f} s, fp64)"}


COPY_BYTES = 256 << 20


def copy_calibration():
    """Three device-to-device copies of COPY_BYTES each (read COPY_BYTES,
    write COPY_BYTES): the reference kernel against which counter readings
    of the GEMMs are scaled to bytes."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").normal_()
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] copy calibration: 3 x {COPY_BYTES >> 20} MiB")


# ------------------------------------------------------------------ main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-extra", action="store_true", help="skip the context workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run three plain 256 MiB device copies, the known-size reference "
                         "for hardware byte counters (FETCH_SIZE / WRITE_SIZE) of the same process")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the layers need no cross-GPU communication on this "
              f"path (--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2404_12406_amd as ms
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    log(f"[bench] {ms.version()} on {torch.cuda.get_device_name(0)}")
    if args.calibrate_copy:
        copy_calibration()
    h = headline(args.steps, args.warmup)
    line = {
        "metric": METRIC,
        "value": round(h["value"], 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(h["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "linear_stack_bf16", "M": 4096, "features": [1024, 4096, 1024, 4096, 1024],
                   "mask": "input+bias per layer, weights frozen", "flop_per_step": h["flop_step"]},
        "saved_activation_bytes": {"selective": h["saved"]["selective"], "all_true": h["saved"]["all_true"]},
        "roofline": h["roofline"],
    }
    if not args.no_extra:
        line["extra"] = extras(args.steps, args.warmup)
    if not args.no_cpu:
        log("[bench] cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline()
        log(f"[bench] cpu baseline {line['cpu_baseline']}")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
