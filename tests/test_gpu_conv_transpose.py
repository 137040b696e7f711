"""GPU parity of the transposed convolution (ConvTranspose2d, and the 1-D
case as H = 1) against the oracle for every mask, in fp32 and bf16, on
geometries that cover overlapping taps, kernels equal to and smaller than
the stride (output pixels no tap reaches get the bias alone), output
padding, channel counts that are not multiples of 8 and several tiles."""
import numpy as np
import pytest

import oracle
import paper_2404_12406_amd as ms
import synth
from oracle import policy as P

from _gpu import check, dev, guarded_empty, guards_intact, host

pytestmark = pytest.mark.gpu

CASES = [
    # x shape, C_out, (R, S), stride, pad, out_pad, dtype
    ((2, 16, 7, 9), 24, (4, 4), (2, 2), (1, 1), (0, 0), "bf16"),     # overlapping taps, 4 phases
    ((2, 24, 6, 5), 16, (2, 2), (2, 2), (0, 0), (0, 0), "bf16"),     # kernel = stride: disjoint stamps
    ((1, 16, 5, 6), 3, (4, 4), (2, 2), (1, 1), (1, 1), "bf16"),      # 3 output channels: padded path
    ((1, 20, 5, 4), 12, (3, 3), (3, 3), (0, 0), (2, 2), "bf16"),     # C_in, C_out not multiples of 8
    ((2, 136, 4, 4), 40, (3, 3), (2, 2), (1, 1), (1, 1), "bf16"),    # several k tiles
    ((2, 64, 16, 16), 32, (3, 3), (1, 1), (1, 1), (0, 0), "bf16"),   # size-preserving, several m tiles
    ((1, 8, 5, 5), 8, (1, 1), (3, 2), (0, 0), (2, 1), "bf16"),       # kernel < stride: holes
    ((2, 8, 9, 7), 8, (3, 3), (1, 1), (1, 1), (0, 0), "f32"),        # the App. B probe layer, small
    ((2, 5, 6, 6), 7, (5, 5), (2, 2), (2, 2), (1, 1), "f32"),
    ((1, 8, 1, 50), 8, (1, 3), (1, 1), (0, 1), (0, 0), "f32"),       # 1-D as H = 1
    ((3, 16, 1, 37), 24, (1, 4), (1, 2), (0, 1), (0, 1), "bf16"),    # 1-D, strided
]


def _inputs(case, seed):
    xs, co, k, st, pd, op, dt = CASES[case]
    ws = (xs[1], co, k[0], k[1])
    x = synth.normal(xs, seed, dtype=dt)
    w = synth.kaiming_uniform(ws, seed + 1, co * k[0] * k[1], dtype=dt)
    b = synth.normal((co,), seed + 2, 0.1, dtype=dt)
    return x, w, b


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("mask", range(8))
def test_conv_transpose_all_masks(case, mask):
    xs, co, k, st, pd, op, dt = CASES[case]
    seed = 8000 + 10 * case
    x, w, b = _inputs(case, seed)
    y_ref = oracle.round_to(oracle.convt2d_forward(x, w, b, st, pd, op), dt)
    gy = synth.normal(y_ref.shape, seed + 3, dtype=dt)
    y, rec = ms.layer_forward(ms.ConvTranspose2d(st, pd, op), dev(x, dt), dev(w, dt), dev(b, dt), mask)
    assert tuple(y.shape) == y_ref.shape
    check("y", host(y), y_ref, dt)
    if mask == 0:
        assert rec is None
        return
    acct = rec.account()
    assert acct["saved_activation_bytes"] == P.saved_activation_bytes("conv_transpose2d", mask, x.size, dt)
    gx, gw, gb = ms.layer_backward(rec, dev(gy, dt))
    assert (gx is not None) == bool(mask & 1)
    assert (gw is not None) == bool(mask & 2)
    assert (gb is not None) == bool(mask & 4)
    if gx is not None:
        check("dx", host(gx), oracle.convt2d_input_grad(gy, w, xs, st, pd, op), dt)
    if gw is not None:
        check("dW", host(gw), oracle.convt2d_weight_grad(gy, x, w.shape, st, pd, op), dt)
    if gb is not None:
        check("db", host(gb), oracle.convt2d_bias_grad(gy), dt)
    rec.free()


@pytest.mark.parametrize("case", [0, 2, 3, 8])
def test_conv_transpose_without_bias_and_output_guards(case):
    """No bias: the forward adds nothing; every output lands inside its own
    buffer (guard bands around y, dx and dW stay untouched)."""
    xs, co, k, st, pd, op, dt = CASES[case]
    x, w, _ = _inputs(case, 8500 + case)
    y_ref = oracle.round_to(oracle.convt2d_forward(x, w, None, st, pd, op), dt)
    y, ybuf, g = guarded_empty(y_ref.shape, dt)
    _, rec = ms.layer_forward(ms.ConvTranspose2d(st, pd, op), dev(x, dt), dev(w, dt), None, 3, y=y)
    check("y", host(y), y_ref, dt)
    assert guards_intact(ybuf, g)
    gy = synth.normal(y_ref.shape, 8600 + case, dtype=dt)
    gx, gxbuf, g1 = guarded_empty(xs, dt)
    gw, gwbuf, g2 = guarded_empty(w.shape, dt)
    ms.layer_backward(rec, dev(gy, dt), grad_x=gx, grad_W=gw)
    check("dx", host(gx), oracle.convt2d_input_grad(gy, w, xs, st, pd, op), dt)
    check("dW", host(gw), oracle.convt2d_weight_grad(gy, x, w.shape, st, pd, op), dt)
    assert guards_intact(gxbuf, g1) and guards_intact(gwbuf, g2)


def test_conv_transpose_is_the_adjoint_of_the_library_convolution():
    """<convT(x), z> = <x, conv(z)> with both sides computed by the library
    (fp32), and each against the oracle."""
    xs, co, k, st, pd, op, dt = CASES[8]
    x, w, _ = _inputs(8, 8700)
    y, _ = ms.layer_forward(ms.ConvTranspose2d(st, pd, op), dev(x, dt), dev(w, dt), None, 0)
    z = synth.normal(tuple(y.shape), 8701, dtype=dt)
    cz, _ = ms.layer_forward(ms.Conv2d(st, pd), dev(z, dt), dev(w, dt), None, 0)
    lhs, rhs = float(np.vdot(host(y), z)), float(np.vdot(x, host(cz)))
    assert abs(lhs - rhs) <= 1e-4 * (abs(lhs) + abs(rhs) + 1.0)


def test_conv_transpose_empty_batch():
    xs = (0, 16, 5, 5)
    x = np.zeros(xs, np.float32)
    w = synth.normal((16, 8, 3, 3), 1, dtype="bf16")
    b = synth.normal((8,), 2, dtype="bf16")
    y, rec = ms.layer_forward(ms.ConvTranspose2d(2, 1, 1), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    assert tuple(y.shape) == (0, 8, 10, 10)
    gy = np.zeros((0, 8, 10, 10), np.float32)
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    assert gx.shape == (0, 16, 5, 5)
    assert float(host(gw).__abs__().max()) == 0.0 and float(host(gb).__abs__().max()) == 0.0
