"""Pins of the conv2d oracle against things other than itself:
scipy's correlate2d/convolve2d (independent library routines), hand-worked
values, adjoint identities, exact central differences of an affine map,
linearity, and special cases that reduce to the linear layer or the identity.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy import signal

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def scipy_conv_fwd(x, w, b, stride, pad):
    """Cross-correlation via scipy.signal.correlate2d on the zero-padded input,
    then subsampled by the stride."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    xp = np.pad(x, ((0, 0), (0, 0), (pad[0], pad[0]), (pad[1], pad[1])))
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    y = np.zeros((N, K, P, Q))
    for n in range(N):
        for k in range(K):
            acc = 0
            for c in range(C):
                acc = acc + signal.correlate2d(xp[n, c], w[k, c], mode="valid")
            y[n, k] = acc[::stride[0], ::stride[1]][:P, :Q] + (b[k] if b is not None else 0)
    return y


def _dilate(dy, stride):
    N, K, P, Q = dy.shape
    out = np.zeros((N, K, (P - 1) * stride[0] + 1, (Q - 1) * stride[1] + 1))
    out[:, :, ::stride[0], ::stride[1]] = dy
    return out


def scipy_conv_dgrad(dy, w, x_shape, stride, pad):
    """Transposed convolution: zero-insert dy by the stride, full 2-D
    convolution with each kernel slice, crop the padding."""
    N, C, H, W = x_shape
    K, _, R, S = w.shape
    du = _dilate(dy, stride)
    dx = np.zeros((N, C, H + 2 * pad[0], W + 2 * pad[1]))
    for n in range(N):
        for c in range(C):
            acc = 0
            for k in range(K):
                acc = acc + signal.convolve2d(du[n, k], w[k, c], mode="full")
            hh = min(acc.shape[0], dx.shape[2])
            ww = min(acc.shape[1], dx.shape[3])
            dx[n, c, :hh, :ww] = acc[:hh, :ww]
    return dx[:, :, pad[0]:pad[0] + H, pad[1]:pad[1] + W]


def scipy_conv_wgrad(dy, x, w_shape, stride, pad):
    K, C, R, S = w_shape
    xp = np.pad(x, ((0, 0), (0, 0), (pad[0], pad[0]), (pad[1], pad[1])))
    du = _dilate(dy, stride)
    dw = np.zeros(w_shape)
    for k in range(K):
        for c in range(C):
            acc = 0
            for n in range(x.shape[0]):
                acc = acc + signal.correlate2d(xp[n, c], du[n, k], mode="valid")
            dw[k, c] = acc[:R, :S]
    return dw


conv_cases = st.tuples(
    st.integers(1, 2),             # N
    st.integers(1, 3),             # C
    st.integers(1, 3),             # K
    st.integers(1, 7),             # H
    st.integers(1, 7),             # W
    st.sampled_from([1, 2, 3, 7]),  # R
    st.sampled_from([1, 2, 3]),     # S
    st.integers(1, 3),             # stride
    st.integers(0, 3),             # pad
    st.integers(0, 2**31 - 1),     # seed
)


def _valid(c):
    N, C, K, H, W, R, S, st_, pd, _ = c
    return H + 2 * pd >= R and W + 2 * pd >= S


def _mk(c):
    N, C, K, H, W, R, S, st_, pd, seed = c
    x = _rand((N, C, H, W), seed)
    w = _rand((K, C, R, S), seed + 1)
    b = _rand((K,), seed + 2)
    stride = (st_, 1 if st_ == 3 else st_)
    pad = (pd, max(0, pd - 1))
    if W + 2 * pad[1] < S:
        pad = (pd, pd)
    return x, w, b, stride, pad


@settings(max_examples=60, deadline=None)
@given(conv_cases.filter(_valid))
def test_forward_matches_scipy_correlate(c):
    x, w, b, stride, pad = _mk(c)
    if x.shape[3] + 2 * pad[1] < w.shape[3]:
        return
    y = oracle.conv2d_forward(x, w, b, stride, pad)
    ref = scipy_conv_fwd(x, w, b, stride, pad)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


@settings(max_examples=60, deadline=None)
@given(conv_cases.filter(_valid))
def test_input_grad_matches_scipy_transposed(c):
    x, w, b, stride, pad = _mk(c)
    if x.shape[3] + 2 * pad[1] < w.shape[3]:
        return
    y = oracle.conv2d_forward(x, w, None, stride, pad)
    dy = _rand(y.shape, c[-1] + 7)
    dx = oracle.conv2d_input_grad(dy, w, x.shape, stride, pad)
    ref = scipy_conv_dgrad(dy, w, x.shape, stride, pad)
    np.testing.assert_allclose(dx, ref, rtol=1e-12, atol=1e-12)


@settings(max_examples=60, deadline=None)
@given(conv_cases.filter(_valid))
def test_weight_grad_matches_scipy(c):
    x, w, b, stride, pad = _mk(c)
    if x.shape[3] + 2 * pad[1] < w.shape[3]:
        return
    y = oracle.conv2d_forward(x, w, None, stride, pad)
    dy = _rand(y.shape, c[-1] + 9)
    dw = oracle.conv2d_weight_grad(dy, x, w.shape, stride, pad)
    ref = scipy_conv_wgrad(dy, x, w.shape, stride, pad)
    np.testing.assert_allclose(dw, ref, rtol=1e-12, atol=1e-12)


@settings(max_examples=80, deadline=None)
@given(conv_cases.filter(_valid))
def test_adjoint_identities(c):
    """<dy, conv(x;W)> = <dgrad(dy;W), x> = <wgrad(dy,x), W>; <dy, 1(x)b> = <db, b>."""
    x, w, b, stride, pad = _mk(c)
    if x.shape[3] + 2 * pad[1] < w.shape[3]:
        return
    y = oracle.conv2d_forward(x, w, None, stride, pad)
    dy = _rand(y.shape, c[-1] + 11)
    lhs = float(np.sum(dy * y))
    dx = oracle.conv2d_input_grad(dy, w, x.shape, stride, pad)
    dw = oracle.conv2d_weight_grad(dy, x, w.shape, stride, pad)
    scale = max(1.0, float(np.sum(np.abs(dy) * np.abs(y))))
    assert abs(lhs - float(np.sum(dx * x))) <= 1e-12 * scale
    assert abs(lhs - float(np.sum(dw * w))) <= 1e-12 * scale
    yb = oracle.conv2d_forward(np.zeros_like(x), w, b, stride, pad)
    db = oracle.conv2d_bias_grad(dy)
    assert abs(float(np.sum(dy * yb)) - float(np.sum(db * b))) <= 1e-12 * max(1.0, float(np.sum(np.abs(dy))))


@settings(max_examples=40, deadline=None)
@given(conv_cases.filter(_valid))
def test_central_differences_exact(c):
    """The layer is affine in x, in W and in b, so (f(t+hv) - f(t-hv)) / 2h
    equals the directional derivative for any h; with h = 1 the VJPs must
    satisfy <dy, Jv> = <vjp(dy), v>."""
    x, w, b, stride, pad = _mk(c)
    if x.shape[3] + 2 * pad[1] < w.shape[3]:
        return
    f = lambda xx, ww, bb: oracle.conv2d_forward(xx, ww, bb, stride, pad)
    y = f(x, w, b)
    dy = _rand(y.shape, c[-1] + 13)
    vx, vw, vb = _rand(x.shape, c[-1] + 14), _rand(w.shape, c[-1] + 15), _rand(b.shape, c[-1] + 16)
    jx = (f(x + vx, w, b) - f(x - vx, w, b)) / 2
    jw = (f(x, w + vw, b) - f(x, w - vw, b)) / 2
    jb = (f(x, w, b + vb) - f(x, w, b - vb)) / 2
    gx = oracle.conv2d_input_grad(dy, w, x.shape, stride, pad)
    gw = oracle.conv2d_weight_grad(dy, x, w.shape, stride, pad)
    gb = oracle.conv2d_bias_grad(dy)
    for j, g, v in ((jx, gx, vx), (jw, gw, vw), (jb, gb, vb)):
        a, bb_ = float(np.sum(dy * j)), float(np.sum(g * v))
        assert abs(a - bb_) <= 1e-10 * max(1.0, abs(a))


def test_linearity_in_x_and_w():
    rng = np.random.default_rng(3)
    x1, x2 = rng.standard_normal((2, 3, 9, 8)), rng.standard_normal((2, 3, 9, 8))
    w1, w2 = rng.standard_normal((4, 3, 3, 2)), rng.standard_normal((4, 3, 3, 2))
    a, bt = 1.7, -0.3
    for stride, pad in (((1, 1), (1, 0)), ((2, 3), (2, 1))):
        f = lambda x, w: oracle.conv2d_forward(x, w, None, stride, pad)
        np.testing.assert_allclose(f(a * x1 + bt * x2, w1), a * f(x1, w1) + bt * f(x2, w1), atol=1e-12)
        np.testing.assert_allclose(f(x1, a * w1 + bt * w2), a * f(x1, w1) + bt * f(x1, w2), atol=1e-12)


def test_pointwise_conv_equals_linear():
    """A 1x1 / stride 1 / pad 0 conv is the linear layer applied to every
    pixel's channel vector; two independent oracle routines must agree."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 5, 4, 6))
    w = rng.standard_normal((7, 5, 1, 1))
    b = rng.standard_normal(7)
    y = oracle.conv2d_forward(x, w, b)
    X = x.transpose(0, 2, 3, 1).reshape(-1, 5)
    Y = oracle.linear_forward(X, w[:, :, 0, 0], b)
    np.testing.assert_allclose(y.transpose(0, 2, 3, 1).reshape(-1, 7), Y, atol=1e-12)
    dy = rng.standard_normal(y.shape)
    dY = dy.transpose(0, 2, 3, 1).reshape(-1, 7)
    dx = oracle.conv2d_input_grad(dy, w, x.shape)
    np.testing.assert_allclose(dx.transpose(0, 2, 3, 1).reshape(-1, 5),
                               oracle.linear_input_grad(dY, w[:, :, 0, 0]), atol=1e-12)
    dw = oracle.conv2d_weight_grad(dy, x, w.shape)
    np.testing.assert_allclose(dw[:, :, 0, 0], oracle.linear_weight_grad(dY, X), atol=1e-12)
    np.testing.assert_allclose(oracle.conv2d_bias_grad(dy), oracle.linear_bias_grad(dY), atol=1e-12)


def test_centre_delta_is_identity():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 4, 5, 7))
    w = np.zeros((4, 4, 3, 3))
    for k in range(4):
        w[k, k, 1, 1] = 1.0
    np.testing.assert_array_equal(oracle.conv2d_forward(x, w, None, (1, 1), (1, 1)), x)


def test_all_ones_interior():
    rng = np.random.default_rng(7)
    w = rng.standard_normal((3, 2, 3, 3))
    b = rng.standard_normal(3)
    y = oracle.conv2d_forward(np.ones((1, 2, 6, 6)), w, b, (1, 1), (1, 1))
    interior = y[0, :, 1:-1, 1:-1]
    expect = w.reshape(3, -1).sum(1) + b
    np.testing.assert_allclose(interior, np.broadcast_to(expect[:, None, None], interior.shape), atol=1e-12)


def test_stride1_input_grad_is_flipped_forward():
    """For stride 1, dgrad = forward conv of dy with the spatially flipped,
    channel-swapped kernel and padding R-1-p."""
    rng = np.random.default_rng(8)
    x_shape = (2, 3, 7, 6)
    w = rng.standard_normal((4, 3, 3, 2))
    pad = (1, 0)
    y = oracle.conv2d_forward(np.zeros(x_shape), w, None, (1, 1), pad)
    dy = rng.standard_normal(y.shape)
    dx = oracle.conv2d_input_grad(dy, w, x_shape, (1, 1), pad)
    wf = w[:, :, ::-1, ::-1].transpose(1, 0, 2, 3)
    ref = oracle.conv2d_forward(dy, wf, None, (1, 1), (3 - 1 - pad[0], 2 - 1 - pad[1]))
    np.testing.assert_allclose(dx, ref, atol=1e-12)


def test_hand_worked_golden():
    g = json.load(open(os.path.join(GOLD, "conv2d_hand.json")))
    x, w, b = np.array(g["x"], float), np.array(g["W"], float), np.array(g["b"], float)
    for case in g["cases"]:
        y = oracle.conv2d_forward(x, w, b, tuple(case["stride"]), tuple(case["pad"]))
        np.testing.assert_array_equal(y, np.array(case["y"], float))


@pytest.mark.parametrize("stride,pad,R", [((1, 1), (1, 1), 3), ((2, 2), (3, 3), 7), ((2, 2), (1, 1), 3),
                                          ((3, 2), (0, 1), 2)])
def test_sampled_entries_match_full(stride, pad, R):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 3, 11, 10))
    w = rng.standard_normal((4, 3, R, R))
    b = rng.standard_normal(4)
    y = oracle.conv2d_forward(x, w, b, stride, pad)
    dy = rng.standard_normal(y.shape)
    idx = np.array(np.unravel_index(np.arange(y.size), y.shape)).T
    np.testing.assert_allclose(oracle.conv2d_forward_at(x, w, b, stride, pad, idx), y.ravel(), atol=1e-12)
    dx = oracle.conv2d_input_grad(dy, w, x.shape, stride, pad)
    idx = np.array(np.unravel_index(np.arange(dx.size), dx.shape)).T
    # the gathered form shares no loop with the scattered one
    np.testing.assert_allclose(oracle.conv2d_input_grad_at(dy, w, x.shape, stride, pad, idx), dx.ravel(), atol=1e-12)
    dw = oracle.conv2d_weight_grad(dy, x, w.shape, stride, pad)
    idx = np.array(np.unravel_index(np.arange(dw.size), dw.shape)).T
    np.testing.assert_allclose(oracle.conv2d_weight_grad_at(dy, x, w.shape, stride, pad, idx), dw.ravel(), atol=1e-12)


def test_ragged_stride_leaves_trailing_rows_zero():
    """When (H + 2p - R) is not a multiple of the stride the last input rows
    feed no output and must get exactly zero input gradient."""
    rng = np.random.default_rng(10)
    x_shape = (1, 2, 8, 8)
    w = rng.standard_normal((3, 2, 3, 3))
    stride, pad = (3, 3), (0, 0)   # P = (8-3)//3 + 1 = 2: rows 6, 7 unused
    y = oracle.conv2d_forward(np.zeros(x_shape), w, None, stride, pad)
    dx = oracle.conv2d_input_grad(rng.standard_normal(y.shape), w, x_shape, stride, pad)
    assert np.all(dx[:, :, 6:, :] == 0) and np.all(dx[:, :, :, 6:] == 0)
    assert np.any(dx[:, :, :6, :6] != 0)
