"""Pins of the 3-D convolution and transposed-convolution oracles (App. B
probes torch.nn.Conv3d and ConvTranspose3d): torch's conv3d /
conv_transpose3d in float64 (forward and autograd gradients), the reduction
to the separately pinned 2-D oracles when the depth axis is trivial, the
adjoint relation between the two layers, and the bilinear identities."""
import numpy as np
import pytest
import torch

import oracle

GEOMS = [
    # x shape, W shape (conv: K,C,T,R,S), stride, pad
    ((2, 3, 5, 4, 6), (4, 3, 3, 2, 3), (1, 1, 1), (1, 0, 1)),
    ((1, 2, 6, 5, 5), (3, 2, 2, 3, 3), (2, 1, 2), (0, 1, 1)),
    ((2, 2, 4, 4, 3), (2, 2, 3, 1, 1), (3, 2, 1), (1, 0, 0)),
]
TGEOMS = [
    # x shape, W shape (Ci,Co,T,R,S), stride, pad, out_pad
    ((2, 3, 3, 4, 2), (3, 4, 3, 2, 3), (1, 1, 1), (1, 0, 1), (0, 0, 0)),
    ((1, 2, 3, 3, 4), (2, 3, 2, 3, 3), (2, 1, 2), (0, 1, 1), (1, 0, 1)),
    ((1, 2, 2, 3, 3), (2, 2, 1, 1, 1), (3, 2, 1), (0, 0, 0), (2, 1, 0)),
]


def _r(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("i", range(len(GEOMS)))
def test_conv3d_matches_torch(i):
    xs, ws, st, pd = GEOMS[i]
    x, w, b = _r(xs, i), _r(ws, 10 + i), _r((ws[0],), 20 + i)
    tx, tw, tb = (torch.tensor(a, requires_grad=True) for a in (x, w, b))
    ty = torch.nn.functional.conv3d(tx, tw, tb, stride=st, padding=pd)
    np.testing.assert_allclose(oracle.conv3d_forward(x, w, b, st, pd), ty.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = _r(tuple(ty.shape), 30 + i)
    ty.backward(torch.from_numpy(dy))
    np.testing.assert_allclose(oracle.conv3d_input_grad(dy, w, xs, st, pd), tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.conv3d_weight_grad(dy, x, ws, st, pd), tw.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.bias_grad5(dy), tb.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("i", range(len(TGEOMS)))
def test_convt3d_matches_torch(i):
    xs, ws, st, pd, op = TGEOMS[i]
    x, w, b = _r(xs, 40 + i), _r(ws, 50 + i), _r((ws[1],), 60 + i)
    tx, tw, tb = (torch.tensor(a, requires_grad=True) for a in (x, w, b))
    ty = torch.nn.functional.conv_transpose3d(tx, tw, tb, stride=st, padding=pd, output_padding=op)
    np.testing.assert_allclose(oracle.convt3d_forward(x, w, b, st, pd, op), ty.detach().numpy(), rtol=1e-12,
                               atol=1e-12)
    dy = _r(tuple(ty.shape), 70 + i)
    ty.backward(torch.from_numpy(dy))
    np.testing.assert_allclose(oracle.convt3d_input_grad(dy, w, xs, st, pd, op), tx.grad.numpy(), rtol=1e-12,
                               atol=1e-12)
    np.testing.assert_allclose(oracle.convt3d_weight_grad(dy, x, ws, st, pd, op), tw.grad.numpy(), rtol=1e-12,
                               atol=1e-12)


def test_trivial_depth_reduces_to_the_2d_oracles():
    """D = T = 1: the 3-D layers are the 2-D ones (pinned on their own)."""
    x, w = _r((2, 3, 1, 5, 6), 80), _r((4, 3, 1, 3, 2), 81)
    np.testing.assert_allclose(oracle.conv3d_forward(x, w, None, (1, 2, 1), (0, 1, 0))[:, :, 0],
                               oracle.conv2d_forward(x[:, :, 0], w[:, :, 0], None, (2, 1), (1, 0)), rtol=1e-13)
    wt = _r((3, 4, 1, 3, 2), 82)
    np.testing.assert_allclose(oracle.convt3d_forward(x, wt, None, (1, 2, 1), (0, 1, 0), (0, 1, 0))[:, :, 0],
                               oracle.convt2d_forward(x[:, :, 0], wt[:, :, 0], None, (2, 1), (1, 0), (1, 0)),
                               rtol=1e-13)


@pytest.mark.parametrize("i", range(len(TGEOMS)))
def test_transposed_is_the_adjoint_and_identities_hold(i):
    xs, ws, st, pd, op = TGEOMS[i]
    x, w = _r(xs, 90 + i), _r(ws, 91 + i)
    y = oracle.convt3d_forward(x, w, None, st, pd, op)
    z = _r(y.shape, 92 + i)
    cz = oracle.conv3d_forward(z, w, None, st, pd)      # W read as [K = Ci, C = Co, T, R, S]
    assert cz.shape == x.shape
    lhs = np.vdot(y, z)
    assert np.isclose(lhs, np.vdot(x, cz), rtol=1e-12)
    assert np.isclose(lhs, np.vdot(x, oracle.convt3d_input_grad(z, w, xs, st, pd, op)), rtol=1e-12)
    assert np.isclose(lhs, np.vdot(w, oracle.convt3d_weight_grad(z, x, ws, st, pd, op)), rtol=1e-12)
