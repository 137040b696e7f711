#!/usr/bin/env python3
"""Benchmark of the selective-differentiation layers on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Headline step: the bf16 Linear layers of a 12-layer hidden-768 transformer
encoder on 16 x 512 tokens (QKV 768->2304, out 768->768, FFN 768->3072->768 per
layer, 48 Linear layers), every weight and bias frozen and gradients flowing to
the inputs only -- the fine-tuning mask of the paper's transformer experiments
(Sec. 3.3).  One step is the forward of all 48 layers and their input
gradients: 96 GEMMs, no weight-gradient GEMM (the mask skips it), through the
C ABI of libmemsave.so.  `value` is the algorithmic TFLOP/s of the launched
contractions over K back-to-back steps with every input resident in HBM.

The same line carries, for the headline and for every other synthetic
workload:
  * the timing protocol: K reps, each after a 512 MiB read sweep that evicts
    the last-level cache, as median / p10 / p90, next to the warm
    back-to-back figure;
  * the shader clock sampled while the steps run;
  * retained activation bytes under the selective rule (read from the
    library's ledger) and, from the library's policy accounting, under stock
    PyTorch's rule and under an all-true mask;
  * a per-layer roofline: each contraction's and each BN pass's own kernel
    time (library HIP events on the launch stream, cache evicted before every
    launch) against min(dense bf16 peak, arithmetic intensity x HBM peak);
and the roofline of the headline's dominant kernel, the HBM bytes the
hardware counters recorded for it, and the CPU oracle timed on a bounded
sample of the headline workload (plus a sampled oracle time per workload).

One JSON line goes to stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import platform
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "conv/linear fwd+bwd TFLOP/s (frozen W) + saved-activation bytes vs full AD"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 (matrix and vector)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
FLUSH_BYTES = 512 << 20        # read sweep that evicts the 256 MB last-level cache
HEADLINE = "encoder_linears_bf16"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


def elt(dtype: str) -> int:
    return 2 if dtype == "bf16" else 4


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


def layer_passes(spec, mask: int, dtype: str):
    """The timed kernels of one layer call: (name, profiling kind, FLOP,
    algorithmic HBM bytes).  A contraction's bytes are its three operands
    read or written once (x, W, y for the forward; dy, W, dx for the input
    gradient; dy, x, dW for the weight gradient).  A transposed
    convolution's forward is an input-gradient contraction and its input
    gradient a forward one (the profiling kinds name the contraction).
    BN-eval: the forward reads x and writes y; the backward reads dy, writes
    dx when asked and reads x when dgamma is asked."""
    import paper_2404_12406_amd as ms
    e = elt(dtype)
    out = []
    if spec.kind in ("conv2d", "linear", "conv_transpose2d"):
        f = layer_flops(spec, mask)
        xb, yb = numel(spec.in_shape) * e, numel(spec.out_shape()) * e
        wb = numel(spec.weight_shape()) * e
        tr = spec.kind == "conv_transpose2d"
        out.append(("forward", ms.PROF_DGRAD if tr else ms.PROF_FWD, f["fwd"], xb + wb + yb))
        if mask & 1:
            out.append(("input_grad", ms.PROF_FWD if tr else ms.PROF_DGRAD, f["dgrad"], yb + wb + xb))
        if mask & 2:
            out.append(("weight_grad", ms.PROF_WGRAD, f["wgrad"], yb + xb + wb))
    elif spec.kind == "bn_eval":
        n = numel(spec.in_shape) * e
        out.append(("forward", ms.PROF_BN, 0, 2 * n))
        if mask:
            out.append(("backward", ms.PROF_RED, 0, n * (1 + (mask & 1) + ((mask >> 1) & 1))))
    return out


def roof(flop: int, nbytes: int, us: float, dtype: str) -> dict:
    """Achieved rate of one timed kernel against its own roofline bound."""
    sec = us * 1e-6
    if flop:
        peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_FP32_TFLOPS
        ai = flop / nbytes
        bound = min(peak, ai * PEAK_HBM_GBS / 1e3)
        ach = flop / sec / 1e12
        return {"tflops": round(ach, 1), "ai_flop_per_byte": round(ai, 1), "bound_tflops": round(bound, 1),
                "bound": "mfma" if bound >= peak else "hbm", "frac_of_bound": round(ach / bound, 4)}
    gbs = nbytes / sec / 1e9
    return {"GBs": round(gbs, 1), "bound": "hbm", "frac_of_bound": round(gbs / PEAK_HBM_GBS, 4)}


def pct(v, q):
    """q-th percentile of v (linear interpolation)."""
    s = sorted(v)
    if len(s) == 1:
        return s[0]
    x = (len(s) - 1) * q / 100.0
    i = int(x)
    j = min(i + 1, len(s) - 1)
    return s[i] + (s[j] - s[i]) * (x - i)


# ------------------------------------------------------------------ cache eviction, clock
class Flusher:
    """A 512 MiB read sweep on the current stream: after it, none of a step's
    operands are left in the last-level cache or the L2s.  (A write sweep
    would leave dirty lines whose write-back competes with the timed work.)"""

    def __init__(self):
        import torch
        self.big = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")

    def __call__(self):
        self.big.sum()


class ClockSampler:
    """Samples the GPU's current shader-clock level from sysfs
    (pp_dpm_sclk of the device's PCI function) every few milliseconds while
    armed; reports the levels seen, weighted by samples."""

    def __init__(self):
        self.path = None
        try:
            import torch
            p = torch.cuda.get_device_properties(0)
            cand = f"/sys/bus/pci/devices/{p.pci_domain_id:04x}:{p.pci_bus_id:02x}:{p.pci_device_id:02x}.0/pp_dpm_sclk"
            if os.access(cand, os.R_OK):
                self.path = cand
        except Exception:
            self.path = None
        if self.path is None:
            c = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
            if len(c) == 1 and os.access(c[0], os.R_OK):
                self.path = c[0]
        self.samples = []
        self._stop = None
        self._th = None

    def _read(self):
        try:
            with open(self.path) as f:
                for line in f:
                    if "*" in line:
                        return int("".join(ch for ch in line.split(":", 1)[1] if ch.isdigit()))
        except Exception:
            return None
        return None

    def start(self):
        if not self.path:
            return
        self._stop = threading.Event()

        def run():
            while not self._stop.is_set():
                v = self._read()
                if v:
                    self.samples.append(v)
                time.sleep(0.002)
        self._th = threading.Thread(target=run, daemon=True)
        self._th.start()

    def stop(self) -> dict:
        if self._th:
            self._stop.set()
            self._th.join()
        if not self.samples:
            return {"source": self.path, "mhz": None}
        s = self.samples
        return {"source": "sysfs pp_dpm_sclk (current DPM level, sampled every 2 ms)", "samples": len(s),
                "median_mhz": statistics.median(s), "min_mhz": min(s), "max_mhz": max(s)}


# ------------------------------------------------------------------ one workload
def build(w):
    from synth import draw, gpu
    arrays = draw.chains(w)
    return arrays, gpu.build_chains(arrays, w.dtype)


def run_steps(chains, n, backward=True):
    for _ in range(n):
        for c in chains:
            c.forward()
        if backward:
            for c in chains:
                c.backward()


def policy_bytes(chains) -> dict:
    """Retained activation bytes of one forward of the chains under the
    three rules, from the library's own policy accounting (every record of
    a forward is alive at its end, so the forward peak is their sum)."""
    import paper_2404_12406_amd as ms
    tot = {"selective": 0, "pytorch_default": 0, "all_true": 0}
    for c in chains:
        for p, lc in zip(c.prepared, c.calls):
            x, W, b = p.tensors[:3]
            for name, pol in (("selective", ms.POLICY_SELECTIVE), ("pytorch_default", ms.POLICY_PYTORCH_DEFAULT),
                              ("all_true", ms.POLICY_ALL_TRUE)):
                tot[name] += ms.policy_account(lc.spec, x, W, b, lc.mask, pol)["saved_activation_bytes"]
    return tot


def ledger_peak_of_forward(chains):
    """Peak retained activation bytes over one forward of `chains`, read from
    the library's ledger."""
    import torch
    import paper_2404_12406_amd as ms
    torch.cuda.synchronize()
    live0, _ = ms.ledger_read()
    ms.ledger_reset()
    for c in chains:
        c.forward()
    torch.cuda.synchronize()
    _, peak = ms.ledger_read()
    for c in chains:
        c.backward()
    torch.cuda.synchronize()
    return peak - live0


def timing(chains, steps, warmup, flush, backward=True, clock=None):
    """K back-to-back steps between one event pair (warm), then K reps each
    after a cache-evicting sweep (cold), each rep between its own events."""
    import torch
    run_steps(chains, warmup, backward)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if clock:
        clock.start()
    wall0 = time.perf_counter()
    e0.record()
    run_steps(chains, steps, backward)
    e1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - wall0) * 1e3 / steps
    warm = e0.elapsed_time(e1) / steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        flush()
        a.record()
        run_steps(chains, 1, backward)
        b.record()
    torch.cuda.synchronize()
    clk = clock.stop() if clock else None
    cold = [a.elapsed_time(b) for a, b in ev]
    return {"warm_ms_per_step": round(warm, 4), "host_wall_ms_per_step": round(wall, 4),
            "cold": {"reps": steps, "median_ms": round(statistics.median(cold), 4), "p10_ms": round(pct(cold, 10), 4),
                     "p90_ms": round(pct(cold, 90), 4)}, "clock": clk}


def per_layer_roofline(chains, w, reps, flush, order=None):
    """Each layer's timed kernels, cache evicted before every launch: the
    layer's forward, then its backward, `reps` times, with every profiling
    kind armed (a layer's forward and backward kernels are of distinct
    kinds).  Layers of identical shape and mask are measured once."""
    import torch
    import paper_2404_12406_amd as ms
    out, seen = [], set()
    specs = iter(w.layers)
    for c in chains:
        for p in c.prepared:
            spec = next(specs)
            passes = layer_passes(spec, p.mask, w.dtype)
            key = (spec.kind, spec.in_shape, spec.out_ch, spec.ksize, spec.stride, spec.pad, p.mask)
            if not passes or key in seen:
                continue
            seen.add(key)
            if order is not None:
                order.append({"layer": spec.name, "mask": p.mask, "reps": reps})
            ms.profile_start(ms.PROF_ALL)
            for _ in range(reps):
                flush()
                p.forward()
                if p.mask:
                    flush()
                    p.backward()
            torch.cuda.synchronize()
            got = {k: ms.profile_read(k) for k in {k for _, k, _, _ in passes}}
            ms.profile_start(0)
            for name, kind, flop, nbytes in passes:
                n, tot = got[kind]
                if n == 0:
                    continue
                us = tot / reps * 1e3   # the call's kernels (a contraction may take two launches)
                e = {"layer": spec.name, "pass": name, "launches_per_call": n // reps, "us": round(us, 2),
                     "flop": flop, "bytes": nbytes}
                e.update(roof(flop, nbytes, us, w.dtype))
                out.append(e)
    return out


def measure(w, steps, warmup, flush, per_layer=True, reps=None):
    import torch
    t0 = time.time()
    _, chains = build(w)
    fl = [layer_flops(l, l.mask) for l in w.layers]
    flop = sum(f["fwd"] + f["dgrad"] + f["wgrad"] for f in fl)
    tm = timing(chains, steps, warmup, flush)
    sel = ledger_peak_of_forward(chains)
    pol = policy_bytes(chains)
    assert sel == pol["selective"], (w.name, sel, pol)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
    warm = tm["warm_ms_per_step"]
    out = {"gflop": round(flop / 1e9, 3), "ms_per_step": warm, "tflops": round(flop / (warm * 1e-3) / 1e12, 2),
           "frac_of_peak": round(flop / (warm * 1e-3) / 1e12 / peak, 4), "timing": tm,
           "cold_tflops_median": round(flop / (tm["cold"]["median_ms"] * 1e-3) / 1e12, 2),
           "saved_activation_bytes": {"selective_ledger": sel, "pytorch_default": pol["pytorch_default"],
                                      "all_true": pol["all_true"]}}
    if per_layer:
        out["per_layer"] = per_layer_roofline(chains, w, reps or min(steps, 20), flush)
    del chains
    torch.cuda.empty_cache()
    log(f"[bench] {w.name}: {warm:.4f} ms/step warm, cold median {tm['cold']['median_ms']:.4f} ms, "
        f"{out['tflops']} TFLOP/s, saved {out['saved_activation_bytes']} ({time.time() - t0:.1f}s)")
    return out


# ------------------------------------------------------------------ recorded counters
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_encoder_linears_bf16_hbm_counters.md")
GEMM_SOURCES = ("paper_2404_12406_amd/csrc/kernels/gemm_bf16.hip", "paper_2404_12406_amd/csrc/kernels/gemm_block_body.inc",
                "paper_2404_12406_amd/csrc/kernels/common.h", "paper_2404_12406_amd/csrc/kernels/limits.h")


def gemm_sources_sha256():
    h = hashlib.sha256()
    for p in GEMM_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(key: str):
    """HBM bytes per layer call of the forward ("fwd") or input-gradient
    ("dgrad") GEMMs of the headline workload from the committed FETCH_SIZE /
    WRITE_SIZE counter summary, or None when the GEMM sources changed since
    the counters were taken (or the summary is absent)."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    fields = dict(l.split(": ", 1) for l in text.splitlines() if ": " in l and not l.startswith(("|", "#", " ")))
    if fields.get("kernel_sources_sha256", "").strip() != gemm_sources_sha256():
        return None
    v = fields.get(f"traffic_bytes_per_call_{key}")
    return int(v) if v else None


# ------------------------------------------------------------------ headline
def headline(steps, warmup, flush):
    import torch
    import paper_2404_12406_amd as ms
    from synth import workloads as wl
    w = wl.encoder_linears_bf16()
    t0 = time.time()
    arrays, chains = build(w)
    fl = [layer_flops(l, l.mask) for l in w.layers]
    flop_step = sum(f["fwd"] + f["dgrad"] + f["wgrad"] for f in fl)
    log(f"[bench] headline {w.name}: {flop_step / 1e9:.1f} GFLOP per step, {len(w.layers)} layers "
        f"(inputs drawn in {time.time() - t0:.1f}s); warmup {warmup}")
    clock = ClockSampler()
    # Pass 1, the headline (warm) and the cold reps: no per-launch
    # instrumentation inside.
    tm = timing(chains, steps, warmup, flush, clock=clock)
    ms_step = tm["warm_ms_per_step"]
    value = flop_step / (ms_step * 1e-3) / 1e12
    # Pass 2, the roofline: K steps again with the library bracketing each
    # forward / input-gradient GEMM launch with HIP events on the stream it
    # launches on.  The dominant kernel is the contraction with the larger
    # summed GPU time.
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms.profile_start(ms.PROF_FWD | ms.PROF_DGRAD)
    ev0.record()
    run_steps(chains, steps)
    ev1.record()
    torch.cuda.synchronize()
    ms_prof = ev0.elapsed_time(ev1) / steps
    kern = {}
    for name, kind, key in (("forward", ms.PROF_FWD, "fwd"), ("input-gradient", ms.PROF_DGRAD, "dgrad")):
        n, tot = ms.profile_read(kind)
        kern[key] = {"name": name, "key": key, "launches": n, "ms": tot, "flop": sum(f[key] for f in fl) * steps}
    ms.profile_start(0)
    dom = max(kern.values(), key=lambda k: k["ms"])
    # one contraction per layer call: one launch, or two where the output's
    # columns are split between two tiles (a partly empty last wave)
    calls = steps * len(w.layers)
    assert calls <= dom["launches"] <= 2 * calls, dom
    achieved = dom["flop"] / (dom["ms"] * 1e-3) / 1e12
    for k in kern.values():
        log(f"[bench]   {k['name']} GEMMs: {k['launches']} launches in {calls} calls, avg {k['ms'] / calls * 1e3:.1f} us "
            f"per call, {k['flop'] / max(k['ms'], 1e-9) / 1e9:.1f} TFLOP/s")
    log(f"[bench] headline {ms_step:.4f} ms/step, {value:.1f} TFLOP/s; cold median {tm['cold']['median_ms']:.4f} ms; "
        f"profiled pass {ms_prof:.4f} ms/step; dominant {dom['name']} GEMMs {achieved:.1f} TFLOP/s; clock {tm['clock']}")
    # per-shape breakdown (the four Linear layers of encoder layer 0), cold
    shapes = per_layer_roofline(chains[:3], _first_encoder_layer(w), min(steps, 20), flush)
    sel = ledger_peak_of_forward(chains)
    pol = policy_bytes(chains)
    assert sel == pol["selective"], (sel, pol)
    del chains
    torch.cuda.empty_cache()
    # the all-true mask, run for real: the ledger's forward peak
    full = build(_with_masks(w, _all_true))[1]
    allb = ledger_peak_of_forward(full)
    assert allb == policy_bytes(full)["all_true"], allb
    del full
    torch.cuda.empty_cache()
    return {
        "workload": w, "arrays": arrays, "ms_per_step": ms_step, "value": value, "flop_step": flop_step, "timing": tm,
        "per_shape": shapes,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": recorded_traffic(dom["key"]),
                     "kernel": f"ms::g2::gemm_kernel ({dom['name']} GEMMs of the 48 Linear layers)",
                     "flop_per_call": dom["flop"] // calls, "avg_call_us": round(dom["ms"] / calls * 1e3, 2),
                     "calls": calls, "launches": dom["launches"], "pass_ms_per_step": round(ms_prof, 4),
                     "unit_of_work": "one layer's contraction (its kernel launches summed: one, or two for a "
                                     "column-split output)",
                     "traffic_unit": "HBM bytes per layer call (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"},
        "saved": {"selective_ledger": sel, "pytorch_default": pol["pytorch_default"], "all_true_ledger": allb},
    }


def _first_encoder_layer(w):
    import copy
    w2 = copy.copy(w)
    w2.layers = w.layers[:4]
    return w2


def _with_masks(w, fn):
    import copy
    w2 = copy.deepcopy(w)
    for l in w2.layers:
        l.mask = fn(l)
    return w2


def _all_true(l):
    if l.kind == "avgpool":
        return 1
    return 1 | 2 | (4 if l.has_bias else 0)


# ------------------------------------------------------------------ bandwidth-bound passes
def reduction_bandwidth(steps, warmup, flush):
    """The HBM-bound backward passes at the ResNet-18-shaped stack's stem
    and stage-1 sizes (bf16, channels-last), each launch after a cache
    eviction:
      * BN-eval backward with every flag (dx = dy s, dgamma = sum dy x_hat,
        dbeta = sum dy): reads dy and x, writes dx (3 numel elt bytes);
      * BN-eval backward with dx alone: 2 numel elt;
      * the bias gradient as a standalone column sum (a conv whose mask
        holds the bias bit alone): reads dy (numel elt), plus its finalize.
    Time: the library's HIP events around the reduction pass (reduction
    kernel and finalize kernels together)."""
    import torch
    import paper_2404_12406_amd as ms
    import synth
    from synth import gpu
    out = []
    for label, shape in (("stem_output", (64, 64, 112, 112)), ("stage1", (64, 64, 56, 56))):
        C = shape[1]
        n = numel(shape)
        x = gpu.dev(synth.normal(shape, 4100, dtype="bf16"), "bf16")
        gy = gpu.dev(synth.normal(shape, 4101, dtype="bf16"), "bf16")
        g_ = gpu.dev(synth.uniform((C,), 4102, 0.5, 1.5, dtype="bf16"), "bf16")
        be = gpu.dev(synth.normal((C,), 4103, 0.1, dtype="bf16"), "bf16")
        mu = gpu.dev(synth.normal((C,), 4104, 0.1, dtype="bf16"), "bf16")
        var = gpu.dev(synth.uniform((C,), 4105, 0.5, 1.5, dtype="bf16"), "bf16")
        spec = ms.BatchNormEval(mu, var, 1e-5)
        cases = []
        for mask, nbytes in ((7, 3 * n * 2), (1, 2 * n * 2)):
            gx = torch.empty_like(x)
            p = ms.PreparedLayer(spec, x, g_, be, mask, grad_y=gy, grad_x=gx if mask & 1 else None,
                                 grad_W=torch.empty_like(g_) if mask & 2 else None,
                                 grad_b=torch.empty_like(be) if mask & 4 else None)
            cases.append((f"bn_eval_backward_mask{mask}", p, nbytes))
        # bias-only conv: its backward is the column sum alone (x is the
        # conv's input, y the shape above)
        xin = torch.zeros((shape[0], 8, shape[2], shape[3]), dtype=torch.bfloat16, device="cuda").contiguous(
            memory_format=torch.channels_last)
        wc = torch.zeros((C, 8, 1, 1), dtype=torch.bfloat16, device="cuda").contiguous(memory_format=torch.channels_last)
        bc = torch.zeros((C,), dtype=torch.bfloat16, device="cuda")
        p = ms.PreparedLayer(ms.Conv2d(1, 0), xin, wc, bc, 4, grad_y=gy, grad_b=torch.empty_like(bc))
        cases.append(("bias_grad_column_sum", p, n * 2))
        for name, p, nbytes in cases:
            for _ in range(max(1, warmup)):
                p.forward()
                p.backward()
            torch.cuda.synchronize()
            ms.profile_start(ms.PROF_RED)
            for _ in range(steps):
                p.forward()
                flush()
                p.backward()
            torch.cuda.synchronize()
            cnt, tot = ms.profile_read(ms.PROF_RED)
            ms.profile_start(0)
            assert cnt == steps, (name, cnt)
            us = tot / cnt * 1e3
            e = {"case": name, "tensor": label, "shape": list(shape), "bytes": nbytes, "us": round(us, 2)}
            e.update(roof(0, nbytes, us, "bf16"))
            out.append(e)
            log(f"[bench] {name} on {label}: {us:.1f} us, {e['GBs']} GB/s")
        del cases, p
    torch.cuda.empty_cache()
    return out


def layout_staging_cost(steps, warmup, flush):
    """What a caller's NCHW tensors cost against channels-last ones: the
    conv sweep's 3x3 layer x[32,256,28,28] with every flag set (forward,
    input, weight and bias gradients) and the BN-eval forward on the stage-1
    tensor [64,64,56,56], bf16, each call after a cache eviction.  For the
    conv in NCHW the library stages x, W, y (and grad_y, grad_x, grad_W)
    through transient workspace with its strided-copy kernel, whose bytes
    (each staged tensor read and written once) are reported beside the
    times; BN-eval sweeps a plain NCHW tensor in place."""
    import torch
    import paper_2404_12406_amd as ms
    out = {}
    g = torch.Generator(device="cuda").manual_seed(4646)
    cl = torch.channels_last
    cases = []
    x = torch.randn(32, 256, 28, 28, generator=g, device="cuda").to(torch.bfloat16)
    w = (0.02 * torch.randn(256, 256, 3, 3, generator=g, device="cuda")).to(torch.bfloat16)
    b = torch.zeros(256, device="cuda", dtype=torch.bfloat16)
    gy = torch.randn(32, 256, 28, 28, generator=g, device="cuda").to(torch.bfloat16)
    # staged tensors, each read and written once: x (forward and weight
    # gradient), y, grad_y, grad_x; W (forward and input gradient), grad_W
    staged = 2 * 2 * (5 * x.numel() + 3 * w.numel())
    for fmt in ("channels_last", "nchw"):
        conv = (lambda t: t.contiguous(memory_format=cl)) if fmt == "channels_last" else (lambda t: t.contiguous())
        X, W, GY = conv(x), conv(w), conv(gy)
        p = ms.PreparedLayer(ms.Conv2d(1, 1), X, W, b, 7, y=conv(torch.empty_like(x)), grad_y=GY,
                             grad_x=conv(torch.empty_like(x)), grad_W=conv(torch.empty_like(w)),
                             grad_b=torch.empty_like(b))
        cases.append(("conv3x3_256_all_flags", fmt, p, staged))
    xb = torch.randn(64, 64, 56, 56, generator=g, device="cuda").to(torch.bfloat16)
    C = 64
    mu, var = torch.zeros(C, device="cuda", dtype=torch.bfloat16), torch.ones(C, device="cuda", dtype=torch.bfloat16)
    ga, be = torch.ones(C, device="cuda", dtype=torch.bfloat16), torch.zeros(C, device="cuda", dtype=torch.bfloat16)
    for fmt in ("channels_last", "nchw"):
        X = xb.contiguous(memory_format=cl) if fmt == "channels_last" else xb.contiguous()
        p = ms.PreparedLayer(ms.BatchNormEval(mu, var, 1e-5), X, ga, be, 0, y=torch.empty_like(X))
        cases.append(("bn_eval_forward_stage1", fmt, p, 0))   # plain NCHW: swept in place, nothing staged
    for name, fmt, p, sbytes in cases:
        for _ in range(max(1, warmup)):
            p.forward()
            if p.mask:
                p.backward()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for a, c in ev:
            flush()
            a.record()
            p.forward()
            if p.mask:
                p.backward()
            c.record()
        torch.cuda.synchronize()
        t = statistics.median(a.elapsed_time(c) for a, c in ev)
        out.setdefault(name, {})[fmt] = {"median_ms": round(t, 4)}
        if fmt == "nchw":
            base = out[name]["channels_last"]["median_ms"]
            out[name]["nchw"].update({"overhead_ms": round(t - base, 4), "staged_bytes": sbytes})
            if sbytes:
                out[name]["nchw"]["staging_GBs"] = round(sbytes / max(t - base, 1e-6) / 1e6, 1)
        log(f"[bench] layout {name} {fmt}: {t:.4f} ms")
    torch.cuda.empty_cache()
    return out


def relu_bandwidth(steps, warmup, flush):
    """ReLU with a 1-bit saved mask (Sec. 2.2.2) on the stem-output tensor of
    the ResNet-18-shaped stack (64 x 64 x 112 x 112 bf16, channels-last).
    HBM bytes per launch: forward reads x and writes y and the mask
    (2 * 2 * n + n / 8), backward reads dy and the mask and writes dx (the
    same).  Each launch is timed by the library's HIP events after a cache
    eviction.  Retained bytes: this library's mask, the paper's one-byte
    boolean mask, stock PyTorch's saved output."""
    import torch
    import paper_2404_12406_amd as ms
    shape = (64, 64, 112, 112)
    n = numel(shape)
    g = torch.Generator(device="cuda").manual_seed(4242)
    x = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    gy = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    gx = torch.empty_like(x)
    p = ms.PreparedLayer(ms.ReLU(), x, mask=ms.MASK_INPUT, grad_y=gy, grad_x=gx)
    for _ in range(max(1, warmup)):
        p.forward()
        p.backward()
    torch.cuda.synchronize()
    nbytes = 2 * 2 * n + n // 8
    out = {"shape": list(shape), "dtype": "bf16", "bytes_per_launch": nbytes}
    ms.profile_start(ms.PROF_ACT)
    for _ in range(steps):
        flush()
        p.forward()
    torch.cuda.synchronize()
    cnt, t_fwd = ms.profile_read(ms.PROF_ACT)
    assert cnt == steps, (cnt, steps)
    ms.profile_start(ms.PROF_ACT)
    for _ in range(steps):
        flush()
        p.forward()
        flush()
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
    return out


def dropout_bandwidth(steps, warmup, flush):
    """Dropout that draws its mask again in backward (Sec. 2.2.2) on the
    stem-output tensor of the ResNet-18-shaped stack (64 x 64 x 112 x 112
    bf16, channels-last) and on the FFN hidden activation of the encoder
    (8192 x 3072 bf16), p = 0.1.  HBM bytes per launch: read the input, write
    the output (2 * 2 * n); no mask is read or written.  ALU work per
    launch: one Philox4x32-10 block per 4 elements.  Each launch is timed by
    the library's HIP events after a cache eviction.  Retained bytes: this
    library keeps the generator state (0 bytes), stock PyTorch a one-byte
    mask (n)."""
    import torch
    import paper_2404_12406_amd as ms
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
            flush()
            p.forward()
        torch.cuda.synchronize()
        cnt, t_fwd = ms.profile_read(ms.PROF_ACT)
        assert cnt == steps, (cnt, steps)
        ms.profile_start(ms.PROF_ACT)
        for _ in range(steps):
            flush()
            p.forward()
            flush()
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


def extras(steps, warmup, flush):
    from synth import workloads as wl
    out = {}
    jobs = [("single_conv2d_f32", wl.single_conv_f32()),
            ("linear_stack_bf16", wl.linear_stack_bf16()),
            ("resnet18_shaped_bf16", wl.resnet18_shaped_bf16()),
            ("resnet18_shaped_bf16_input", wl.resnet18_shaped_bf16(input_requires_grad=True)),
            ("decoder_convt_bf16", wl.decoder_convt_bf16())]
    for mk in ("00", "10", "01", "11"):
        jobs.append((f"conv_sweep_3x3_{mk}", wl.conv_sweep_bf16(mk)))
        jobs.append((f"conv_sweep_1x1_{mk}", wl.conv_sweep_bf16(mk, pointwise=True)))
    for name, w in jobs:
        out[name] = measure(w, steps, warmup, flush)
    t0 = time.time()
    out["reduction_passes"] = reduction_bandwidth(steps, warmup, flush)
    log(f"[bench] reduction passes ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["layout_staging"] = layout_staging_cost(min(steps, 20), warmup, flush)
    log(f"[bench] layout staging ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["fig1_synthetic_cnn_memory"] = f1 = memory_probe("conv2d")
    log(f"[bench] fig1 probe: library {f1['library']}, stock {f1['stock_pytorch']} ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["conv3d_training_step_bf16"] = c3 = conv3d_throughput(min(steps, 10), warmup)
    log(f"[bench] 3-D convolutions: {c3} ({time.time() - t0:.1f}s)")
    out["appB_layer_memory"] = {}
    for kind in ("conv_transpose2d", "conv1d", "conv_transpose1d", "conv3d", "conv_transpose3d"):
        t0 = time.time()
        out["appB_layer_memory"][kind] = pr = memory_probe(kind)
        log(f"[bench] App. B probe {kind}: library {pr['library']}, stock {pr['stock_pytorch']} "
            f"({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["dropout_regenerated_mask"] = dr = dropout_bandwidth(min(steps, 20), warmup, flush)
    log(f"[bench] dropout: " + ", ".join(f"{k} fwd {v['forward']} bwd {v['backward']}" for k, v in dr.items())
        + f" ({time.time() - t0:.1f}s)")
    t0 = time.time()
    out["relu_bitmask_stem_output"] = rl = relu_bandwidth(min(steps, 20), warmup, flush)
    log(f"[bench] relu: forward {rl['forward']}, backward {rl['backward']} ({time.time() - t0:.1f}s)")
    return out


# ------------------------------------------------------------------ CPU oracle
def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(arrays, target_s: float = 15.0):
    """The oracle (fp64 C loops, OpenMP) on the first `rows` rows of every
    one of the headline's 48 Linear layers: forward and input gradient of
    each; the rate scales to the whole step by its FLOP count."""
    import oracle

    def run(rows):
        t = time.perf_counter()
        for ca in arrays:
            acts = [ca.x[:rows]]
            for la in ca.layers:
                acts.append(oracle.round_to(oracle.linear_forward(acts[-1], la.W, la.b), "bf16"))
            g = ca.grad_y[:rows]
            for la in reversed(ca.layers):
                g = oracle.round_to(oracle.linear_input_grad(g, la.W), "bf16")
        return time.perf_counter() - t

    per_row = sum(2 * 2 * la.spec.in_shape[1] * la.spec.out_ch for ca in arrays for la in ca.layers)
    # grow the sample until it takes at least half the target (the rate per
    # row rises with the row count, as the loops' threads get more work)
    rows, cap = 2, arrays[0].x.shape[0]
    t = run(rows)
    while t < 0.5 * target_s and rows < cap:
        rows = int(min(cap, rows * min(8.0, max(1.5, target_s / max(t, 1e-3)))))
        t = run(rows)
    return {"value": round(rows * per_row / t / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{rows} of 8192 rows of all 48 layers, fwd+input grad, fp64"}


def oracle_samples(target_s: float = 3.0):
    """A sampled oracle time per workload: the contractions of one step on
    a bounded sample of output entries (rows of the Linear stack; sampled
    output entries of every conv, from inputs of the layer's shape), scaled
    to the step by FLOP count.  Single-conv workload: the whole step."""
    import numpy as np
    import oracle
    import synth
    from synth import workloads as wl
    rng = np.random.default_rng(0)
    out = {}

    # single conv, fp32: whole forward + input gradient
    w = wl.single_conv_f32()
    l = w.layers[0]
    x = synth.normal(l.in_shape, 1, dtype="f32")
    wt = synth.kaiming_uniform(l.weight_shape(), 2, 144)
    gy = synth.normal(l.out_shape(), 3, dtype="f32")
    t = time.perf_counter()
    oracle.conv2d_forward(x, wt, None, l.stride, l.pad)
    oracle.conv2d_input_grad(gy, wt, l.in_shape, l.stride, l.pad)
    dt = time.perf_counter() - t
    f = sum(layer_flops(l, l.mask).values())
    out["single_conv2d_f32"] = {"step_s": round(dt, 4), "GFLOPs": round(f / dt / 1e9, 3), "sample": "whole step"}

    def conv_sampled(w, name, nsample):
        tot_f, tot_t = 0, 0.0
        for l in w.layers:
            if l.kind != "conv2d":
                continue
            xs, ws, ys = l.in_shape, l.weight_shape(), l.out_shape()
            # float64 inputs, so the timed calls convert nothing
            x = rng.standard_normal(xs)
            wt = rng.standard_normal(ws)
            idx = np.stack([rng.integers(0, e, nsample) for e in ys], 1)
            t = time.perf_counter()
            oracle.conv2d_forward_at(x, wt, None, l.stride, l.pad, idx)
            tot_t += time.perf_counter() - t
            tot_f += 2 * nsample * ws[1] * ws[2] * ws[3]
            fl = layer_flops(l, l.mask)
            if fl["dgrad"]:
                gy = rng.standard_normal(ys)
                xi = np.stack([rng.integers(0, e, nsample) for e in xs], 1)
                t = time.perf_counter()
                oracle.conv2d_input_grad_at(gy, wt, xs, l.stride, l.pad, xi)
                tot_t += time.perf_counter() - t
                tot_f += 2 * nsample * ws[0] * ws[2] * ws[3] // (l.stride[0] * l.stride[1])
            if fl["wgrad"]:
                gy = rng.standard_normal(ys)
                wi = np.stack([rng.integers(0, e, max(1, nsample // 64)) for e in ws], 1)
                t = time.perf_counter()
                oracle.conv2d_weight_grad_at(gy, x, ws, l.stride, l.pad, wi)
                tot_t += time.perf_counter() - t
                tot_f += 2 * len(wi) * ys[0] * ys[2] * ys[3]
        step_f = sum(sum(layer_flops(l, l.mask).values()) for l in w.layers)
        rate = tot_f / tot_t
        out[name] = {"GFLOPs": round(rate / 1e9, 3), "step_s_extrapolated": round(step_f / rate, 2),
                     "sample": f"{nsample} sampled outputs per conv contraction ({tot_f / 1e9:.2f} GFLOP in {tot_t:.1f} s)"}

    conv_sampled(wl.resnet18_shaped_bf16(), "resnet18_shaped_bf16", 16384)
    conv_sampled(wl.conv_sweep_bf16("11"), "conv_sweep_3x3_11", 65536)
    # Linear stack: forward + input gradient + bias gradient of the first rows
    w = wl.linear_stack_bf16()
    rows = 64
    X = rng.standard_normal((rows, 1024))
    t = time.perf_counter()
    tot_f = 0
    a = X
    Ws = []
    for l in w.layers:
        W = rng.standard_normal((l.out_ch, l.in_shape[1])) * 0.02
        Ws.append(W)
        a = oracle.linear_forward(a, W)
        tot_f += 2 * rows * l.in_shape[1] * l.out_ch
    g = rng.standard_normal((rows, 1024))
    for W in reversed(Ws):
        oracle.linear_bias_grad(g)
        g = oracle.linear_input_grad(g, W)
        tot_f += 2 * rows * W.shape[0] * W.shape[1]
    dt = time.perf_counter() - t
    step_f = sum(sum(layer_flops(l, l.mask).values()) for l in w.layers)
    out["linear_stack_bf16"] = {"GFLOPs": round(tot_f / dt / 1e9, 3), "step_s_extrapolated": round(step_f / (tot_f / dt), 2),
                                "sample": f"first {rows} of 4096 rows"}
    return out


# ------------------------------------------------------------------ counters
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
def workload_by_name(name):
    from synth import workloads as wl
    table = {"single_conv2d_f32": wl.single_conv_f32, "linear_stack_bf16": wl.linear_stack_bf16,
             "resnet18_shaped_bf16": wl.resnet18_shaped_bf16,
             "resnet18_shaped_bf16_input": lambda: wl.resnet18_shaped_bf16(input_requires_grad=True),
             "encoder_linears_bf16": wl.encoder_linears_bf16, "decoder_convt_bf16": wl.decoder_convt_bf16}
    for mk in ("00", "10", "01", "11"):
        table[f"conv_sweep_3x3_{mk}"] = (lambda m: lambda: wl.conv_sweep_bf16(m))(mk)
        table[f"conv_sweep_1x1_{mk}"] = (lambda m: lambda: wl.conv_sweep_bf16(m, pointwise=True))(mk)
    if name not in table:
        raise SystemExit(f"unknown workload {name!r}; one of {sorted(table)}")
    return table[name]()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle timings")
    ap.add_argument("--workload", default=None,
                    help="measure these workloads only (comma-separated names: warm and cold steps, per-layer "
                         "kernels) and print one record each; for kernel traces and counters")
    ap.add_argument("--per-layer-only", action="store_true",
                    help="with --workload: one untimed step, then only the per-layer kernel timings (every "
                         "layer call preceded by a cache-evicting sweep, so a kernel trace splits at the sweeps)")
    ap.add_argument("--reduction-only", action="store_true",
                    help="only the HBM-bound backward passes (BN-eval backward with every flag and with dx "
                         "alone, the standalone bias column sum) at the stem and stage-1 sizes, each launch "
                         "after a cache-evicting sweep; for kernel traces and counters")
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
    flush = Flusher()
    if args.reduction_only:
        print(json.dumps({"reduction_passes": reduction_bandwidth(args.steps, args.warmup, flush)}), flush=True)
        return
    if args.workload:
        for name in args.workload.split(","):
            w = workload_by_name(name)
            if args.per_layer_only:
                _, chains = build(w)
                run_steps(chains, 1)
                torch.cuda.synchronize()
                order = []
                rec = {"per_layer": per_layer_roofline(chains, w, args.steps, flush, order), "measured": order}
                del chains
                torch.cuda.empty_cache()
            else:
                rec = measure(w, args.steps, args.warmup, flush)
            print(json.dumps({"workload": name, **rec}), flush=True)
        return
    h = headline(args.steps, args.warmup, flush)
    w = h["workload"]
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
        "config": {"workload": HEADLINE, "layers": 12, "tokens": 8192, "hidden": 768,
                   "linears_per_layer": ["768->2304", "768->768", "768->3072", "3072->768"],
                   "mask": "input only, weights and biases frozen", "flop_per_step": h["flop_step"]},
        "saved_activation_bytes": h["saved"],
        "timing": h["timing"],
        "roofline": h["roofline"],
        "per_shape": h["per_shape"],
    }
    if not args.no_extra:
        line["extra"] = extras(args.steps, args.warmup, flush)
    del flush
    if not args.no_cpu:
        log("[bench] cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline(h["arrays"])
        line["cpu_baseline"]["cpu"] = cpu_model()
        line["cpu_baseline"]["nproc"] = os.cpu_count()
        log(f"[bench] cpu baseline {line['cpu_baseline']}")
        line["oracle_samples"] = oracle_samples()
        log(f"[bench] oracle samples {line['oracle_samples']}")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
