"""GPU parity of every layer kind and mask against the oracle, on seeded
inputs at sizes that span several tiles and end in ragged tails.  Every call
goes through the C ABI (libmemsave.so) via the Python binding."""
import gc

import numpy as np
import pytest
import torch

import oracle
import paper_2404_12406_amd as ms
import synth
from oracle import policy as P

from _gpu import TOL, check, dev, guarded_empty, guards_intact, host

pytestmark = pytest.mark.gpu

MASKS = list(range(8))


def _conv_inputs(seed, shape_x, shape_w, dtype, bias=True):
    x = synth.normal(shape_x, seed, dtype=dtype)
    fan_in = shape_w[1] * shape_w[2] * shape_w[3]
    w = synth.kaiming_uniform(shape_w, seed + 1, fan_in, dtype=dtype)
    b = synth.normal((shape_w[0],), seed + 2, 1.0, dtype=dtype) if bias else None   # output scale: a dropped bias fails
    return x, w, b


CONV_CASES = [
    # (x shape, w shape, stride, pad, dtype)
    ((8, 16, 32, 32), (32, 16, 3, 3), (1, 1), (1, 1), "f32"),    # the fp32 single-conv workload
    ((3, 24, 13, 11), (40, 24, 3, 3), (1, 1), (1, 1), "bf16"),
    ((2, 16, 15, 14), (24, 16, 3, 3), (2, 2), (1, 1), "bf16"),
    ((2, 3, 30, 29), (16, 3, 7, 7), (2, 2), (3, 3), "bf16"),      # stem-like, C=3 scalar path
    ((2, 32, 9, 10), (48, 32, 1, 1), (1, 1), (0, 0), "bf16"),     # pointwise (GEMM path)
    ((2, 16, 9, 10), (24, 16, 1, 1), (2, 2), (0, 0), "bf16"),     # strided 1x1: odd phases get no taps
    ((1, 12, 11, 13), (20, 12, 3, 2), (3, 2), (0, 1), "bf16"),    # C, K not multiples of 8
    ((2, 8, 7, 9), (8, 8, 3, 3), (1, 1), (1, 1), "f32"),
    ((2, 5, 12, 12), (7, 5, 5, 5), (2, 1), (2, 1), "f32"),
    ((1, 8, 5, 5), (136, 8, 3, 3), (1, 1), (0, 0), "bf16"),       # several N tiles
]


@pytest.mark.parametrize("case", range(len(CONV_CASES)))
@pytest.mark.parametrize("mask", MASKS)
def test_conv2d_all_masks(case, mask):
    xs, ws, stride, pad, dt = CONV_CASES[case]
    seed = 100 + 10 * case
    x, w, b = _conv_inputs(seed, xs, ws, dt)
    y_ref = oracle.round_to(oracle.conv2d_forward(x, w, b, stride, pad), dt)
    assert oracle.rel_err(oracle.conv2d_forward(x, w, None, stride, pad), y_ref) > 10 * TOL[dt]
    gy = synth.normal(y_ref.shape, seed + 3, dtype=dt)
    X, Wt, B = dev(x, dt), dev(w, dt), dev(b, dt)
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), X, Wt, B, mask)
    check("y", host(y), y_ref, dt)
    if mask == 0:
        assert rec is None
        return
    acct = rec.account()
    assert acct["saved_activation_bytes"] == P.saved_activation_bytes("conv2d", mask, x.size, dt)
    gx, gw, gb = ms.layer_backward(rec, dev(gy, dt))
    assert (gx is not None) == bool(mask & 1)
    assert (gw is not None) == bool(mask & 2)
    assert (gb is not None) == bool(mask & 4)
    if gx is not None:
        check("dx", host(gx), oracle.conv2d_input_grad(gy, w, x.shape, stride, pad), dt)
    if gw is not None:
        check("dW", host(gw), oracle.conv2d_weight_grad(gy, x, w.shape, stride, pad), dt)
    if gb is not None:
        check("db", host(gb), oracle.conv2d_bias_grad(gy), dt)
    rec.free()


LINEAR_CASES = [
    (300, 72, 136, "bf16"),
    (64, 512, 1000, "bf16"),     # classifier head of the ResNet-18-shaped stack
    (129, 30, 20, "bf16"),       # K_in not a multiple of 8: scalar loads
    (200, 48, 72, "f32"),
    (1, 8, 8, "bf16"),
]


@pytest.mark.parametrize("case", range(len(LINEAR_CASES)))
@pytest.mark.parametrize("mask", MASKS)
def test_linear_all_masks(case, mask):
    M, Kin, Nout, dt = LINEAR_CASES[case]
    seed = 300 + 10 * case
    x = synth.normal((M, Kin), seed, dtype=dt)
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype=dt)
    b = synth.normal((Nout,), seed + 2, 1.0, dtype=dt)     # output scale: a dropped bias fails the bar
    gy = synth.normal((M, Nout), seed + 3, dtype=dt)
    y, rec = ms.layer_forward(ms.Linear(), dev(x, dt), dev(w, dt), dev(b, dt), mask)
    y_ref = oracle.linear_forward(x, w, b)
    assert oracle.rel_err(oracle.linear_forward(x, w, None), y_ref) > 10 * TOL[dt]
    check("y", host(y), y_ref, dt)
    if mask == 0:
        assert rec is None
        return
    assert rec.account()["saved_activation_bytes"] == P.saved_activation_bytes("linear", mask, x.size, dt)
    gx, gw, gb = ms.layer_backward(rec, dev(gy, dt))
    if mask & 1:
        check("dX", host(gx), oracle.linear_input_grad(gy, w), dt)
    if mask & 2:
        check("dW", host(gw), oracle.linear_weight_grad(gy, x), dt)
    if mask & 4:
        check("db", host(gb), oracle.linear_bias_grad(gy), dt)


BN_CASES = [
    ((3, 24, 7, 9), "bf16", True),
    ((3, 24, 7, 9), "f32", True),
    ((2, 13, 5, 6), "bf16", True),     # C not a multiple of 8: scalar path
    ((50, 36), "f32", True),           # [N, C] input
    ((4, 64, 9, 9), "bf16", False),    # affine=False
    ((2, 512, 7, 7), "bf16", True),
    # channels-last sweeps whose row of vectors divides 256 (a block streams one
    # contiguous range): 256 vectors per row in bf16 and in f32, 4 f32 vectors,
    # 2 scalar channels, and one 8-channel vector over 3 pixels
    ((2, 2048, 3, 5), "bf16", True),
    ((3, 1024, 2, 3), "f32", True),
    ((5, 16, 3, 3), "f32", True),
    ((3, 2, 5, 7), "bf16", True),
    ((1, 8, 1, 3), "bf16", True),
]


@pytest.mark.parametrize("case", range(len(BN_CASES)))
@pytest.mark.parametrize("mask", MASKS)
def test_bn_eval_all_masks(case, mask):
    shape, dt, affine = BN_CASES[case]
    if not affine and mask & 6:
        pytest.skip("no gamma/beta without affine")
    C = shape[1]
    seed = 500 + 10 * case
    x = synth.normal(shape, seed, dtype=dt)
    mean = synth.normal((C,), seed + 1, 0.1, dtype=dt)
    var = synth.uniform((C,), seed + 2, 0.5, 1.5, dtype=dt)
    g = synth.uniform((C,), seed + 3, 0.5, 1.5, dtype=dt) if affine else None
    bt = synth.normal((C,), seed + 4, 0.1, dtype=dt) if affine else None
    gy = synth.normal(shape, seed + 5, dtype=dt)
    spec = ms.BatchNormEval(dev(mean, dt), dev(var, dt), 1e-5)
    G = dev(g, dt) if affine else None
    Bt = dev(bt, dt) if affine else None
    y, rec = ms.layer_forward(spec, dev(x, dt), G, Bt, mask)
    check("y", host(y), oracle.bn_eval_forward(x, mean, var, g, bt, 1e-5), dt)
    if mask == 0:
        assert rec is None
        return
    acct = rec.account()
    assert acct["saved_activation_bytes"] == P.saved_activation_bytes("bn_eval", mask, x.size, dt)
    gx, gg, gb = ms.layer_backward(rec, dev(gy, dt))
    rdx, rdg, rdb = oracle.bn_eval_backward(gy, x, mean, var, g, 1e-5)
    if mask & 1:
        check("dx", host(gx), rdx, dt)
    if mask & 2:
        check("dgamma", host(gg), rdg, dt)
    if mask & 4:
        check("dbeta", host(gb), rdb, dt)


@pytest.mark.parametrize("shape,dt", [((4, 40, 7, 7), "bf16"), ((3, 12, 5, 3), "f32"), ((2, 13, 4, 4), "bf16")])
def test_avgpool(shape, dt):
    x = synth.normal(shape, 700, dtype=dt)
    gy = synth.normal(shape[:2], 701, dtype=dt)
    y, rec = ms.layer_forward(ms.AvgPool(), dev(x, dt), None, None, ms.MASK_INPUT)
    check("y", host(y), oracle.avgpool_forward(x), dt)
    assert rec.account()["saved_activation_bytes"] == 0
    gx, _, _ = ms.layer_backward(rec, dev(gy, dt))
    check("dx", host(gx), oracle.avgpool_backward(gy, shape), dt)


def test_outputs_write_nothing_outside():
    """Outputs and gradients live between NaN guard bands that must survive."""
    dt = "bf16"
    xs, ws, stride, pad = (2, 16, 15, 14), (24, 16, 3, 3), (2, 2), (1, 1)
    x, w, b = _conv_inputs(900, xs, ws, dt)
    yshape = ms.output_shape(ms.Conv2d(stride, pad), torch.empty(xs), torch.empty(ws))
    y, ybuf, g = guarded_empty(yshape, dt)
    _, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, dt), dev(w, dt), dev(b, dt), 7, y=y)
    gy = synth.normal(yshape, 901, dtype=dt)
    gx, gxb, _ = guarded_empty(xs, dt)
    gw, gwb, _ = guarded_empty(ws, dt)
    gb, gbb, _ = guarded_empty((ws[0],), dt)
    ms.layer_backward(rec, dev(gy, dt), gx, gw, gb)
    torch.cuda.synchronize()
    for buf in (ybuf, gxb, gwb, gbb):
        assert guards_intact(buf, g)
    check("y", host(y), oracle.round_to(oracle.conv2d_forward(x, w, b, stride, pad), dt), dt)
    check("dx", host(gx), oracle.conv2d_input_grad(gy, w, xs, stride, pad), dt)
    check("dW", host(gw), oracle.conv2d_weight_grad(gy, x, ws, stride, pad), dt)
    check("db", host(gb), oracle.conv2d_bias_grad(gy), dt)


def test_empty_batch_and_zero_features():
    dt = "bf16"
    x = torch.empty((0, 16, 8, 8), dtype=torch.bfloat16, device="cuda").contiguous(memory_format=torch.channels_last)
    w = dev(synth.normal((8, 16, 3, 3), 1, dtype=dt), dt)
    b = dev(synth.normal((8,), 2, dtype=dt), dt)
    y, rec = ms.layer_forward(ms.Conv2d(1, 1), x, w, b, 7)
    assert tuple(y.shape) == (0, 8, 8, 8)
    gy = torch.empty_like(y)
    gx, gw, gb = ms.layer_backward(rec, gy)
    torch.cuda.synchronize()
    assert gx.shape == x.shape
    assert torch.all(gw == 0) and torch.all(gb == 0)
    # zero input features: y = b broadcast, dW is empty, db = column sums
    X = torch.empty((5, 0), dtype=torch.bfloat16, device="cuda")
    W = torch.empty((6, 0), dtype=torch.bfloat16, device="cuda")
    bb = synth.normal((6,), 3, dtype=dt)
    y, rec = ms.layer_forward(ms.Linear(), X, W, dev(bb, dt), 5)
    check("y", host(y), np.broadcast_to(bb, (5, 6)), dt)
    gyy = synth.normal((5, 6), 4, dtype=dt)
    gx, _, gb = ms.layer_backward(rec, dev(gyy, dt))
    check("db", host(gb), gyy.sum(0), dt)
    assert gx.shape == (5, 0)


def test_record_lifecycle_and_ledger():
    dt = "bf16"
    x, w, b = _conv_inputs(1000, (2, 16, 8, 8), (16, 16, 3, 3), dt)
    ms.ledger_reset()
    live0, _ = ms.ledger_read()
    X = dev(x, dt)
    _, rec = ms.layer_forward(ms.Conv2d(1, 1), X, dev(w, dt), dev(b, dt), 6)   # W, B: keeps x
    nbytes = x.size * 2
    live, peak = ms.ledger_read()
    assert live - live0 == nbytes and peak >= live
    assert "x" in rec.saved
    gy = dev(synth.normal((2, 16, 8, 8), 1001, dtype=dt), dt)
    with pytest.raises(ms.MemsaveError) as e:        # grad_x given but INPUT not set
        ms.layer_backward(rec, gy, grad_x=torch.empty_like(X))
    assert e.value.status == 2
    ms.layer_backward(rec, gy)
    live, _ = ms.ledger_read()
    assert live == live0                              # backward released the borrow
    with pytest.raises(ms.MemsaveError) as e:
        ms.layer_backward(rec, gy)
    assert e.value.status == 7                        # consumed
    rec.free()
    rec.free()


def test_frozen_weight_input_is_freed_by_allocator():
    """With the weight frozen the record keeps no reference to x: dropping
    the caller's x returns its bytes to the caching allocator, while a
    weight-trainable record keeps exactly numel*elt bytes alive."""
    dt = "bf16"
    shape = (4, 64, 32, 32)
    w = dev(synth.kaiming_uniform((64, 64, 3, 3), 5, 576, dtype=dt), dt)
    for mask, keeps in ((1, False), (3, True)):
        torch.cuda.synchronize()
        X = dev(synth.normal(shape, 6, dtype=dt), dt)
        y, rec = ms.layer_forward(ms.Conv2d(1, 1), X, w, None, mask)
        torch.cuda.synchronize()
        # memory_allocated() is process-wide: keep the cycle collector from
        # freeing unrelated tensors inside the measured window
        gc.collect()
        gc.disable()
        try:
            before = torch.cuda.memory_allocated()
            del X
            torch.cuda.synchronize()
            after = torch.cuda.memory_allocated()
        finally:
            gc.enable()
        freed = before - after
        nbytes = int(np.prod(shape)) * 2
        assert rec.account()["saved_activation_bytes"] == (nbytes if keeps else 0)
        assert freed == (0 if keeps else nbytes)
        rec.free()


def test_kernel_timing_counts_launches():
    """ms_profile_* brackets exactly the armed contraction launches."""
    x, w, b = _conv_inputs(7, (2, 32, 16, 16), (64, 32, 3, 3), "bf16")
    X, Wt, B = dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16")
    ms.profile_start(ms.PROF_FWD | ms.PROF_DGRAD)
    for _ in range(3):
        y, rec = ms.layer_forward(ms.Conv2d((1, 1), (1, 1)), X, Wt, B, 3)
        ms.layer_backward(rec, torch.ones_like(y))
    nf, tf = ms.profile_read(ms.PROF_FWD)
    nd, td = ms.profile_read(ms.PROF_DGRAD)
    nw, tw = ms.profile_read(ms.PROF_WGRAD)
    ms.profile_start(0)
    assert (nf, nd, nw) == (3, 3, 0)
    assert tf > 0 and td > 0 and tw == 0
    y, rec = ms.layer_forward(ms.Conv2d((1, 1), (1, 1)), X, Wt, B, 0)
    assert ms.profile_read(ms.PROF_FWD) == (0, 0.0)


NARROW_CASES = [
    # x shape, w shape, stride, pad: at most 4 channels with a stride-2 width run
    # as a stride-1 convolution over packed column pairs (the stem's path); with
    # stride 2 in both dimensions the input gradient packs 2 x 2 pixel blocks
    ((2, 3, 30, 29), (16, 3, 7, 7), (2, 2), (3, 3)),     # padded width odd, S odd
    ((2, 3, 28, 28), (24, 3, 7, 7), (2, 2), (3, 3)),     # padded width even, S odd
    ((1, 4, 17, 30), (8, 4, 3, 4), (1, 2), (1, 1)),      # width even, S even
    ((2, 1, 9, 21), (16, 1, 5, 5), (2, 2), (0, 2)),      # one channel
    ((1, 2, 12, 13), (8, 2, 3, 3), (2, 2), (1, 1)),
    ((1, 3, 10, 11), (8, 3, 3, 4), (2, 2), (1, 1)),      # padded width odd, S even: channel padding instead
    ((1, 3, 11, 12), (8, 3, 4, 3), (2, 2), (1, 1)),      # blocks do not fit the height: pairs, two phases
]


@pytest.mark.parametrize("case", range(len(NARROW_CASES)))
@pytest.mark.parametrize("mask", [0, 7, 1, 2])
def test_narrow_inputs_with_stride_two_width(case, mask):
    xs, ws, stride, pad = NARROW_CASES[case]
    seed = 9970 + 10 * case
    x, w, b = _conv_inputs(seed, xs, ws, "bf16")
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), mask)
    check("y", host(y), oracle.conv2d_forward(x, w, b, stride, pad), "bf16")
    if rec is None:
        return
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    if gx is not None:
        check("dx", host(gx), oracle.conv2d_input_grad(gy, w, xs, stride, pad), "bf16")
    if gw is not None:
        check("dW", host(gw), oracle.conv2d_weight_grad(gy, x, ws, stride, pad), "bf16")
    if gb is not None:
        check("db", host(gb), oracle.conv2d_bias_grad(gy), "bf16")
