"""The no-allocation backward (ms_layer_backward_noalloc) against
ms_layer_backward, through the C ABI: the same record inputs, the same
gradients bit for bit, on two calls in a row whose second input is smaller
(the fixed scratch keeps the first call's bytes), for every kind of
workspace the backward uses: bias-gradient partial rows of a Linear input
gradient, split-K partials and bias partials of a weight gradient, the
transposed filter of a strided input gradient, packed copies of a
3-channel input, BN-eval reduction partials.  A backward whose workspace
exceeds the scratch is refused before anything runs and the record stays
usable."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2404_12406_amd as ms
import synth
from paper_2404_12406_amd import _lib
from paper_2404_12406_amd.api import _ptr, _stream, tensor_desc

from _gpu import dev

pytestmark = pytest.mark.gpu


def _record(spec, x, W, b, mask):
    _, rec = ms.layer_forward(spec, x, W, b, mask)
    return rec


def _grads(rec, gy, x, W, b):
    m = rec.mask
    gx = torch.full_like(x, float("nan")) if m & 1 else None
    gw = torch.full_like(W, float("nan")) if m & 2 else None
    gb = torch.full_like(b, float("nan")) if m & 4 else None
    return gx, gw, gb


def _run(entry, rec, gy, gx, gw, gb):
    lib = _lib.load()
    fn = lib.ms_layer_backward_noalloc if entry == "noalloc" else lib.ms_layer_backward
    st = fn(rec._h, _ptr(tensor_desc(gy)), _ptr(tensor_desc(gx)), _ptr(tensor_desc(gw)), _ptr(tensor_desc(gb)),
            _stream(gy.device))
    return st


def _case(kind, big):
    """(spec, x, W, b, mask, grad_y) of one case; `big` picks the first,
    larger call of the pair."""
    s = 7000 + (0 if big else 50)
    if kind == "linear_input_bias":
        M, Ki, No = (1024, 1024, 4096) if big else (200, 512, 1000)
        x = dev(synth.normal((M, Ki), s, dtype="bf16"), "bf16")
        W = dev(synth.normal((No, Ki), s + 1, 0.02, dtype="bf16"), "bf16")
        b = dev(synth.normal((No,), s + 2, 1.0, dtype="bf16"), "bf16")
        spec, mask, ys = ms.Linear(), 5, (M, No)
    elif kind == "conv_weight_bias":
        xs, ws = ((8, 64, 28, 28), (128, 64, 3, 3)) if big else ((2, 32, 14, 13), (64, 32, 3, 3))
        x = dev(synth.normal(xs, s, dtype="bf16"), "bf16")
        W = dev(synth.kaiming_uniform(ws, s + 1, ws[1] * 9, dtype="bf16"), "bf16")
        b = dev(synth.normal((ws[0],), s + 2, 1.0, dtype="bf16"), "bf16")
        spec, mask = ms.Conv2d(1, 1), 6
        ys = (xs[0], ws[0], xs[2], xs[3])
    elif kind == "conv_strided_all":
        xs, ws = ((4, 64, 28, 28), (128, 64, 3, 3)) if big else ((2, 16, 15, 14), (24, 16, 3, 3))
        x = dev(synth.normal(xs, s, dtype="bf16"), "bf16")
        W = dev(synth.kaiming_uniform(ws, s + 1, ws[1] * 9, dtype="bf16"), "bf16")
        b = dev(synth.normal((ws[0],), s + 2, 1.0, dtype="bf16"), "bf16")
        spec, mask = ms.Conv2d(2, 1), 7
        ys = (xs[0], ws[0], (xs[2] + 2 - 3) // 2 + 1, (xs[3] + 2 - 3) // 2 + 1)
    elif kind == "conv_3ch_stem":
        xs = (4, 3, 64, 64) if big else (2, 3, 30, 29)
        ws = (64, 3, 7, 7) if big else (16, 3, 7, 7)
        x = dev(synth.normal(xs, s, dtype="bf16"), "bf16")
        W = dev(synth.kaiming_uniform(ws, s + 1, 147, dtype="bf16"), "bf16")
        b = None
        spec, mask = ms.Conv2d(2, 3), 3
        ys = (xs[0], ws[0], (xs[2] + 6 - 7) // 2 + 1, (xs[3] + 6 - 7) // 2 + 1)
    elif kind == "bn_eval_all":
        xs = (8, 64, 28, 28) if big else (2, 32, 7, 5)
        C = xs[1]
        x = dev(synth.normal(xs, s, dtype="bf16"), "bf16")
        W = dev(synth.uniform((C,), s + 1, 0.5, 1.5, dtype="bf16"), "bf16")
        b = dev(synth.normal((C,), s + 2, 0.1, dtype="bf16"), "bf16")
        mean = dev(synth.normal((C,), s + 3, 0.1, dtype="bf16"), "bf16")
        var = dev(synth.uniform((C,), s + 4, 0.5, 1.5, dtype="bf16"), "bf16")
        spec, mask, ys = ms.BatchNormEval(mean, var, 1e-5), 7, xs
    else:
        raise ValueError(kind)
    gy = dev(synth.normal(ys, s + 5, dtype="bf16"), "bf16")
    return spec, x, W, b, mask, gy


KINDS = ["linear_input_bias", "conv_weight_bias", "conv_strided_all", "conv_3ch_stem", "bn_eval_all"]


@pytest.mark.parametrize("kind", KINDS)
def test_noalloc_backward_matches_backward_on_two_calls(kind):
    for big in (True, False):
        spec, x, W, b, mask, gy = _case(kind, big)
        print(f"[no-alloc] {kind} {'first' if big else 'second'} call x={tuple(x.shape)} mask={mask}", flush=True)
        out = {}
        for entry in ("backward", "noalloc"):
            rec = _record(spec, x, W, b, mask)
            ws = rec.account()["transient_workspace_bytes"]
            assert ws <= _lib.load().ms_noalloc_scratch_bytes()
            gx, gw, gb = _grads(rec, gy, x, W, b)
            st = _run(entry, rec, gy, gx, gw, gb)
            assert st == 0, _lib.load().ms_last_error().decode()
            torch.cuda.synchronize()
            out[entry] = [t.clone() for t in (gx, gw, gb) if t is not None]
            rec.free()
        assert len(out["backward"]) == bin(mask).count("1")
        for a, c in zip(out["backward"], out["noalloc"]):
            assert not torch.isnan(c.float()).any()
            # the same kernels on the same inputs: identical bytes
            assert torch.equal(a.view(torch.int16), c.view(torch.int16)), kind


def test_noalloc_backward_refuses_workspace_beyond_the_scratch():
    """A Conv3d weight gradient whose depth-folded input (3 x 51 MB) does
    not fit the scratch: refused, nothing launched, record intact."""
    lib = _lib.load()
    cap = lib.ms_noalloc_scratch_bytes()
    cl = torch.channels_last_3d
    x = torch.randn(4, 64, 16, 56, 56, device="cuda").to(torch.bfloat16).contiguous(memory_format=cl)
    W = (0.05 * torch.randn(64, 64, 3, 3, 3, device="cuda")).to(torch.bfloat16).contiguous(memory_format=cl)
    b = torch.zeros(64, device="cuda", dtype=torch.bfloat16)
    rec = _record(ms.Conv3d(1, 1), x, W, b, 6)
    need = rec.account()["transient_workspace_bytes"]
    assert need > cap, (need, cap)
    gy = torch.randn(4, 64, 16, 56, 56, device="cuda").to(torch.bfloat16).contiguous(memory_format=cl)
    gx, gw, gb = _grads(rec, gy, x, W, b)
    live0, _ = ms.ledger_read()
    assert _run("noalloc", rec, gy, gx, gw, gb) == _lib.MS_E_UNSUPPORTED
    assert "scratch" in lib.ms_last_error().decode()
    torch.cuda.synchronize()
    assert torch.isnan(gw.float()).all() and torch.isnan(gb.float()).all()   # nothing ran
    assert ms.ledger_read()[0] == live0                                        # the record still holds x
    assert _run("backward", rec, gy, gx, gw, gb) == 0
    torch.cuda.synchronize()
    assert not torch.isnan(gw.float()).any()
    rec.free()
