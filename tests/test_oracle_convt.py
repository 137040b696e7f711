"""Pins of the transposed-convolution oracle against things other than
itself: hand-worked values, scipy's convolve2d (a true 2-D convolution of
the stride-dilated input), torch's conv_transpose2d in float64, the
block-stamp closed form when the stride equals the kernel, the adjoint
relation to the (separately pinned) convolution oracle, and the bilinear
identities that tie the two gradients to the forward."""
import json
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st
from scipy import signal

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def scipy_convt(x, w, b, stride, pad, out_pad):
    """Zero-insert x by the stride, full 2-D convolution with each W[i,o]
    slice, then drop `pad` rows/columns at the top/left; rows past the end of
    the full result (reached only through out_pad) receive the bias alone."""
    N, Ci, H, W = x.shape
    _, Co, R, S = w.shape
    Ho, Wo = oracle.convt2d_out_hw(H, W, R, S, stride, pad, out_pad)
    xd = np.zeros((N, Ci, (H - 1) * stride[0] + 1, (W - 1) * stride[1] + 1))
    xd[:, :, ::stride[0], ::stride[1]] = x
    y = np.zeros((N, Co, Ho, Wo))
    for n in range(N):
        for o in range(Co):
            full = 0
            for i in range(Ci):
                full = full + signal.convolve2d(xd[n, i], w[i, o], mode="full")
            crop = full[pad[0]:pad[0] + Ho, pad[1]:pad[1] + Wo]
            y[n, o, :crop.shape[0], :crop.shape[1]] = crop
            y[n, o] += b[o] if b is not None else 0.0
    return y


def torch_convt(x, w, b, stride, pad, out_pad):
    return torch.nn.functional.conv_transpose2d(
        torch.from_numpy(x), torch.from_numpy(w), None if b is None else torch.from_numpy(b),
        stride=tuple(stride), padding=tuple(pad), output_padding=tuple(out_pad)).numpy()


GEOMS = [
    # x shape, (Ci, Co, R, S), stride, pad, out_pad
    ((2, 3, 5, 4), (3, 4, 3, 3), (1, 1), (0, 0), (0, 0)),
    ((2, 3, 5, 4), (3, 4, 3, 3), (1, 1), (1, 1), (0, 0)),
    ((1, 2, 4, 5), (2, 3, 4, 4), (2, 2), (1, 1), (0, 0)),
    ((1, 2, 4, 5), (2, 3, 3, 3), (2, 2), (1, 1), (1, 1)),
    ((2, 2, 3, 3), (2, 2, 2, 2), (2, 2), (0, 0), (0, 0)),    # stride = kernel: disjoint stamps
    ((1, 3, 3, 4), (3, 2, 1, 1), (3, 2), (0, 0), (2, 1)),    # kernel < stride: holes
    ((1, 2, 4, 3), (2, 2, 5, 3), (3, 1), (2, 1), (1, 0)),
    ((1, 1, 6, 2), (1, 3, 3, 2), (1, 2), (2, 0), (0, 1)),    # pad = R - 1
]


def test_hand_worked_values():
    g = json.load(open(os.path.join(GOLD, "convt2d_hand.json")))
    x, w, b = np.array(g["x"], float), np.array(g["W"], float), np.array(g["b"], float)
    for c in g["cases"]:
        y = oracle.convt2d_forward(x, w, b, c["stride"], c["pad"], c["out_pad"])
        np.testing.assert_array_equal(y, np.array(c["y"], float))


@pytest.mark.parametrize("geom", range(len(GEOMS)))
def test_forward_matches_scipy_and_torch(geom):
    xs, ws, stride, pad, op = GEOMS[geom]
    x, w, b = _rand(xs, 10 + geom), _rand(ws, 20 + geom), _rand((ws[1],), 30 + geom)
    y = oracle.convt2d_forward(x, w, b, stride, pad, op)
    np.testing.assert_allclose(y, scipy_convt(x, w, b, stride, pad, op), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y, torch_convt(x, w, b, stride, pad, op), rtol=1e-12, atol=1e-12)


def test_stride_equal_to_kernel_is_a_block_stamp():
    """Stride = kernel size, no padding: output block (h, w) is
    sum_i x[n,i,h,w] W[i,o] (a Kronecker product per channel pair)."""
    x, w, b = _rand((2, 3, 4, 5), 1), _rand((3, 2, 3, 2), 2), _rand((2,), 3)
    y = oracle.convt2d_forward(x, w, b, (3, 2), (0, 0))
    blocks = np.einsum("nihw,iors->nohrws", x, w).reshape(2, 2, 12, 10) + b[None, :, None, None]
    np.testing.assert_allclose(y, blocks, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("geom", range(len(GEOMS)))
def test_adjoint_of_the_convolution(geom):
    """The transposed convolution is the adjoint of the convolution with the
    same filter read as [K = Ci, C = Co, R, S]: <convT(x), z> = <x, conv(z)>."""
    xs, ws, stride, pad, op = GEOMS[geom]
    x, w = _rand(xs, 40 + geom), _rand(ws, 50 + geom)
    y = oracle.convt2d_forward(x, w, None, stride, pad, op)
    z = _rand(y.shape, 60 + geom)
    cz = oracle.conv2d_forward(z, w, None, stride, pad)
    assert cz.shape == x.shape
    assert np.isclose(np.vdot(y, z), np.vdot(x, cz), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("geom", range(len(GEOMS)))
def test_gradients_match_torch_autograd(geom):
    xs, ws, stride, pad, op = GEOMS[geom]
    x, w, b = _rand(xs, 70 + geom), _rand(ws, 80 + geom), _rand((ws[1],), 90 + geom)
    tx, tw, tb = (torch.tensor(a, requires_grad=True) for a in (x, w, b))
    ty = torch.nn.functional.conv_transpose2d(tx, tw, tb, stride=stride, padding=pad, output_padding=op)
    dy = _rand(tuple(ty.shape), 100 + geom)
    ty.backward(torch.from_numpy(dy))
    np.testing.assert_allclose(oracle.convt2d_input_grad(dy, w, xs, stride, pad, op), tx.grad.numpy(),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.convt2d_weight_grad(dy, x, ws, stride, pad, op), tw.grad.numpy(),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.convt2d_bias_grad(dy), tb.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("geom", range(len(GEOMS)))
def test_bilinear_identities(geom):
    """y is linear in x and in W: <y(x, W), dy> = <x, dx(dy)> = <W, dW(dy, x)>
    (bias 0), which pins both gradients to the forward with no library."""
    xs, ws, stride, pad, op = GEOMS[geom]
    x, w = _rand(xs, 110 + geom), _rand(ws, 120 + geom)
    y = oracle.convt2d_forward(x, w, None, stride, pad, op)
    dy = _rand(y.shape, 130 + geom)
    lhs = np.vdot(y, dy)
    assert np.isclose(lhs, np.vdot(x, oracle.convt2d_input_grad(dy, w, xs, stride, pad, op)), rtol=1e-12)
    assert np.isclose(lhs, np.vdot(w, oracle.convt2d_weight_grad(dy, x, ws, stride, pad, op)), rtol=1e-12)


def test_gradients_are_the_convolution_kernels():
    """The input gradient is the convolution's forward of dy, the weight
    gradient the convolution's weight gradient with x as its output gradient."""
    xs, ws, stride, pad, op = GEOMS[3]
    x, w = _rand(xs, 140), _rand(ws, 141)
    y = oracle.convt2d_forward(x, w, None, stride, pad, op)
    dy = _rand(y.shape, 142)
    np.testing.assert_allclose(oracle.convt2d_input_grad(dy, w, xs, stride, pad, op),
                               oracle.conv2d_forward(dy, w, None, stride, pad), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.convt2d_weight_grad(dy, x, ws, stride, pad, op),
                               oracle.conv2d_weight_grad(x, dy, ws, stride, pad), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("geom", range(len(GEOMS)))
def test_sampled_entries_equal_full(geom):
    xs, ws, stride, pad, op = GEOMS[geom]
    x, w, b = _rand(xs, 150 + geom), _rand(ws, 160 + geom), _rand((ws[1],), 170 + geom)
    y = oracle.convt2d_forward(x, w, b, stride, pad, op)
    dy = _rand(y.shape, 180 + geom)
    rng = np.random.default_rng(geom)
    iy = np.stack([rng.integers(0, e, 20) for e in y.shape], 1)
    np.testing.assert_allclose(oracle.convt2d_forward_at(x, w, b, stride, pad, op, iy), y[tuple(iy.T)], rtol=1e-13)
    dx = oracle.convt2d_input_grad(dy, w, xs, stride, pad, op)
    ix = np.stack([rng.integers(0, e, 20) for e in xs], 1)
    np.testing.assert_allclose(oracle.convt2d_input_grad_at(dy, w, xs, stride, pad, op, ix), dx[tuple(ix.T)],
                               rtol=1e-13, atol=1e-15)
    dw = oracle.convt2d_weight_grad(dy, x, ws, stride, pad, op)
    iw = np.stack([rng.integers(0, e, 20) for e in ws], 1)
    np.testing.assert_allclose(oracle.convt2d_weight_grad_at(dy, x, ws, stride, pad, op, iw), dw[tuple(iw.T)],
                               rtol=1e-13, atol=1e-15)


def test_output_padding_must_be_below_stride():
    with pytest.raises(ValueError):
        oracle.convt2d_out_hw(3, 3, 3, 3, (2, 2), (0, 0), (2, 0))


@settings(max_examples=25, deadline=None)
@given(H=st.integers(1, 5), W=st.integers(1, 5), R=st.integers(1, 4), S=st.integers(1, 4),
       sh=st.integers(1, 3), sw=st.integers(1, 3), ph=st.integers(0, 2), pw=st.integers(0, 2),
       oh=st.integers(0, 2), ow=st.integers(0, 2), seed=st.integers(0, 1000))
def test_random_geometry_against_torch(H, W, R, S, sh, sw, ph, pw, oh, ow, seed):
    oh, ow = min(oh, sh - 1), min(ow, sw - 1)
    Ho, Wo = (H - 1) * sh - 2 * ph + R + oh, (W - 1) * sw - 2 * pw + S + ow
    if Ho < 1 or Wo < 1:
        return
    x, w, b = _rand((1, 2, H, W), seed), _rand((2, 3, R, S), seed + 1), _rand((3,), seed + 2)
    np.testing.assert_allclose(oracle.convt2d_forward(x, w, b, (sh, sw), (ph, pw), (oh, ow)),
                               torch_convt(x, w, b, (sh, sw), (ph, pw), (oh, ow)), rtol=1e-12, atol=1e-12)
