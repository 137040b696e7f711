"""Pins of the oracle's ReLU with a 1-bit saved mask (Sec. 2.2.2): a
hand-worked golden, numpy's packbits, torch's relu and its autograd in
float64, the layout mapping against torch's channels-last memory order,
and the paper's size ratios for the saved mask."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import policy as P

GOLD = os.path.join(os.path.dirname(__file__), "golden", "relu_bits.json")


def _f(v):
    return np.array([float(s) for s in v], dtype=np.float64)


def test_hand_worked_golden():
    g = json.load(open(GOLD))
    x, y, dy, dx = _f(g["x"]), _f(g["y"]), _f(g["dy"]), _f(g["dx"])
    got = oracle.relu_forward(x)
    assert np.array_equal(np.isnan(got), np.isnan(y))
    m = ~np.isnan(y)
    assert np.array_equal(got[m], y[m]) and np.array_equal(np.signbit(got[m]), np.signbit(y[m]))
    assert oracle.relu_mask_bits(x).tolist() == g["bits"]
    assert np.array_equal(oracle.relu_backward(dy, x), dx)


@pytest.mark.parametrize("n", [0, 1, 7, 8, 9, 31, 32, 33, 64, 1000, 4099])
def test_mask_is_packbits_of_positive_outputs(n):
    rng = np.random.default_rng(100 + n)
    x = rng.standard_normal(n)
    x[rng.random(n) < 0.1] = 0.0
    x[::13] = np.nan
    want = np.packbits(~(np.maximum(x, 0) <= 0), bitorder="little")
    want = np.concatenate([want, np.zeros(oracle.relu_mask_nbytes(n) - want.size, np.uint8)])
    assert np.array_equal(oracle.relu_mask_bits(x), want)
    assert oracle.relu_mask_nbytes(n) == P.relu_mask_bytes(n) == (4 * ((n + 31) // 32) if n else 0)


def test_forward_and_backward_match_torch_autograd():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((3, 5, 4, 6))
    x.flat[::11] = 0.0
    x.flat[5] = np.nan
    dy = rng.standard_normal(x.shape)
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    yt = torch.relu(xt)
    (gx,) = torch.autograd.grad(yt, xt, torch.tensor(dy))
    y = oracle.relu_forward(x)
    assert np.array_equal(np.isnan(y), np.isnan(yt.detach().numpy()))
    m = ~np.isnan(y)
    assert np.array_equal(y[m], yt.detach().numpy()[m])
    # torch's relu backward passes the gradient where the output is not <= 0
    # (positive or NaN)
    assert np.array_equal(oracle.relu_backward(dy, x), gx.numpy())


def test_memory_order_is_torch_channels_last():
    a = np.arange(2 * 3 * 4 * 5, dtype=np.float64).reshape(2, 3, 4, 5)
    t = torch.tensor(a).contiguous(memory_format=torch.channels_last)
    mem = torch.as_strided(t, (t.numel(),), (1,)).numpy()
    assert np.array_equal(oracle.memory_order(a, "nhwc"), mem)
    assert np.array_equal(oracle.memory_order(a[0, 0], "plain"), a[0, 0].reshape(-1))


def test_backward_is_the_vjp_of_the_forward():
    # relu is linear on the fixed activation pattern: <dy, J v> = <J^T dy, v>
    rng = np.random.default_rng(3)
    x = rng.standard_normal(257)
    v, dy = rng.standard_normal(257), rng.standard_normal(257)
    pos = ~(oracle.relu_forward(x) <= 0)
    jv = np.where(pos, v, 0.0)
    assert np.dot(dy, jv) == pytest.approx(np.dot(oracle.relu_backward(dy, x), v), rel=1e-14, abs=1e-14)


@pytest.mark.parametrize("dtype,ratio", [("f32", 32), ("bf16", 16)])
def test_saved_mask_size_ratios(dtype, ratio):
    # Sec. 2.2.2: a one-byte boolean mask is 4x smaller than a float32 output,
    # one-bit booleans 32x; stock PyTorch keeps the output itself.
    n = 64 * 112 * 112 * 8
    stock = P.saved_activation_bytes("relu", P.MASK_INPUT, n, dtype, P.PYTORCH_DEFAULT)
    ours = P.saved_activation_bytes("relu", P.MASK_INPUT, n, dtype, P.SELECTIVE)
    assert stock == n * P.ELT[dtype]
    assert stock == ratio * ours
    assert n * 4 == 4 * n * 1            # the paper's one-byte mask against fp32: 4x
    assert P.saved_activation_bytes("relu", 0, n, dtype, P.SELECTIVE) == 0
    assert P.saved_activation_bytes("relu", 0, n, dtype, P.ALL_TRUE) == ours


def test_relu_keeps_the_next_layers_input_free():
    # ReLU feeding a frozen conv, the input requiring grad (Sec. 2.2.2): stock
    # PyTorch keeps the ReLU output, which is the conv input; here the conv
    # keeps nothing (weight frozen) and the ReLU one bit per element.
    n = 64 * 64 * 56 * 56
    layers = [("relu", P.MASK_INPUT, n, "bf16"), ("conv2d", P.MASK_INPUT, n, "bf16", True, False)]
    assert P.stack_saved_bytes(layers, P.SELECTIVE) == n // 8
    assert P.saved_activation_bytes("relu", P.MASK_INPUT, n, "bf16", P.PYTORCH_DEFAULT) == 2 * n
