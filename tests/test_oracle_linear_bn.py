"""Pins of the linear, BN-eval, average-pool and rounding oracles."""
import json
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@settings(max_examples=40, deadline=None)
@given(st.integers(0, 9), st.integers(1, 9), st.integers(1, 9), st.integers(0, 2**31 - 1))
def test_linear_matches_numpy_matmul(M, Kin, Nout, seed):
    rng = np.random.default_rng(seed)
    X, W, b = rng.standard_normal((M, Kin)), rng.standard_normal((Nout, Kin)), rng.standard_normal(Nout)
    dY = rng.standard_normal((M, Nout))
    np.testing.assert_allclose(oracle.linear_forward(X, W, b), X @ W.T + b, atol=1e-12)
    np.testing.assert_allclose(oracle.linear_input_grad(dY, W), dY @ W, atol=1e-12)
    np.testing.assert_allclose(oracle.linear_weight_grad(dY, X), dY.T @ X, atol=1e-12)
    np.testing.assert_allclose(oracle.linear_bias_grad(dY), dY.sum(0), atol=1e-12)


def test_linear_adjoint_and_differences():
    rng = np.random.default_rng(1)
    X, W, b = rng.standard_normal((13, 6)), rng.standard_normal((5, 6)), rng.standard_normal(5)
    G = rng.standard_normal((13, 5))
    Y0 = oracle.linear_forward(X, W, None)
    lhs = np.sum(G * Y0)
    assert abs(lhs - np.sum(oracle.linear_input_grad(G, W) * X)) < 1e-11
    assert abs(lhs - np.sum(oracle.linear_weight_grad(G, X) * W)) < 1e-11
    vX, vW, vb = rng.standard_normal(X.shape), rng.standard_normal(W.shape), rng.standard_normal(5)
    f = oracle.linear_forward
    assert abs(np.sum(G * (f(X + vX, W, b) - f(X - vX, W, b)) / 2) - np.sum(oracle.linear_input_grad(G, W) * vX)) < 1e-10
    assert abs(np.sum(G * (f(X, W + vW, b) - f(X, W - vW, b)) / 2) - np.sum(oracle.linear_weight_grad(G, X) * vW)) < 1e-10
    assert abs(np.sum(G * (f(X, W, b + vb) - f(X, W, b - vb)) / 2) - np.sum(oracle.linear_bias_grad(G) * vb)) < 1e-10


def test_linear_sampled_match_full():
    rng = np.random.default_rng(2)
    X, W, b = rng.standard_normal((17, 9)), rng.standard_normal((11, 9)), rng.standard_normal(11)
    dY = rng.standard_normal((17, 11))
    Y = oracle.linear_forward(X, W, b)
    idx = np.array(np.unravel_index(np.arange(Y.size), Y.shape)).T
    np.testing.assert_allclose(oracle.linear_forward_at(X, W, b, idx), Y.ravel(), atol=1e-12)
    dX = oracle.linear_input_grad(dY, W)
    idx = np.array(np.unravel_index(np.arange(dX.size), dX.shape)).T
    np.testing.assert_allclose(oracle.linear_input_grad_at(dY, W, idx), dX.ravel(), atol=1e-12)
    dW = oracle.linear_weight_grad(dY, X)
    idx = np.array(np.unravel_index(np.arange(dW.size), dW.shape)).T
    np.testing.assert_allclose(oracle.linear_weight_grad_at(dY, X, idx), dW.ravel(), atol=1e-12)


def test_bn_eval_hand_worked_golden():
    g = json.load(open(os.path.join(GOLD, "bn_eval_2ch.json")))
    a = {k: np.array(v, float) for k, v in g.items() if isinstance(v, list)}
    y = oracle.bn_eval_forward(a["x"], a["running_mean"], a["running_var"], a["gamma"], a["beta"], g["eps"])
    np.testing.assert_array_equal(y, a["y"])
    dx, dg, dbt = oracle.bn_eval_backward(a["dy"], a["x"], a["running_mean"], a["running_var"], a["gamma"], g["eps"])
    np.testing.assert_array_equal(dx, a["dx"])
    np.testing.assert_array_equal(dg, a["dgamma"])
    np.testing.assert_array_equal(dbt, a["dbeta"])


def test_bn_eval_identity_case():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 4, 5, 2))
    eps = 0.25
    var = np.full(4, 1 - eps)
    y = oracle.bn_eval_forward(x, np.zeros(4), var, np.ones(4), np.zeros(4), eps)
    np.testing.assert_array_equal(y, x)
    y2 = oracle.bn_eval_forward(x, np.zeros(4), var, None, None, eps)
    np.testing.assert_array_equal(y2, x)


def test_bn_eval_matches_torch_cpu_batch_norm():
    """torch.nn.functional.batch_norm(training=False) on the CPU in float64 is
    an independent library routine for the same formula."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((4, 6, 3, 5))
    mean, var = rng.standard_normal(6) * 0.1, rng.uniform(0.5, 1.5, 6)
    gamma, beta = rng.uniform(0.5, 1.5, 6), rng.standard_normal(6) * 0.1
    ref = torch.nn.functional.batch_norm(torch.tensor(x), torch.tensor(mean), torch.tensor(var),
                                         torch.tensor(gamma), torch.tensor(beta), training=False, eps=1e-5)
    np.testing.assert_allclose(oracle.bn_eval_forward(x, mean, var, gamma, beta, 1e-5), ref.numpy(), atol=1e-12)
    xt = torch.tensor(x, requires_grad=True)
    gt = torch.tensor(gamma, requires_grad=True)
    bt = torch.tensor(beta, requires_grad=True)
    yt = torch.nn.functional.batch_norm(xt, torch.tensor(mean), torch.tensor(var), gt, bt, training=False, eps=1e-5)
    dy = rng.standard_normal(x.shape)
    yt.backward(torch.tensor(dy))
    dx, dg, dbt = oracle.bn_eval_backward(dy, x, mean, var, gamma, 1e-5)
    np.testing.assert_allclose(dx, xt.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(dbt, bt.grad.numpy(), atol=1e-11)


def test_bn_eval_central_differences_and_masking():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((2, 3, 4, 4))
    mean, var = rng.standard_normal(3), rng.uniform(0.5, 1.5, 3)
    g, b = rng.standard_normal(3), rng.standard_normal(3)
    dy = rng.standard_normal(x.shape)
    f = lambda xx, gg, bb: oracle.bn_eval_forward(xx, mean, var, gg, bb, 1e-5)
    dx, dg, dbt = oracle.bn_eval_backward(dy, x, mean, var, g, 1e-5)
    v = [rng.standard_normal(x.shape), rng.standard_normal(3), rng.standard_normal(3)]
    assert abs(np.sum(dy * (f(x + v[0], g, b) - f(x - v[0], g, b)) / 2) - np.sum(dx * v[0])) < 1e-10
    assert abs(np.sum(dy * (f(x, g + v[1], b) - f(x, g - v[1], b)) / 2) - np.sum(dg * v[1])) < 1e-10
    assert abs(np.sum(dy * (f(x, g, b + v[2]) - f(x, g, b - v[2])) / 2) - np.sum(dbt * v[2])) < 1e-10
    # the input gradient needs neither x nor the running mean
    dx2, dg2, db2 = oracle.bn_eval_backward(dy, None, mean * 0 + 123.0, var, g, 1e-5, True, False, False)
    np.testing.assert_array_equal(dx2, dx)
    assert dg2 is None and db2 is None


def test_avgpool_adjoint_and_constant():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((3, 4, 7, 7))
    y = oracle.avgpool_forward(x)
    np.testing.assert_allclose(y, x.mean(axis=(2, 3)), atol=1e-14)
    dy = rng.standard_normal(y.shape)
    dx = oracle.avgpool_backward(dy, x.shape)
    assert abs(np.sum(dy * y) - np.sum(dx * x)) < 1e-12
    np.testing.assert_array_equal(oracle.avgpool_forward(np.full((1, 2, 7, 7), 3.5)), np.full((1, 2), 3.5))


def test_round_bf16_known_values():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties to even -> 1 + 2^-6
    # 1 + 2^-8 + 2^-30 lies just above a tie: rounding straight from float64
    # gives 1 + 2^-7 (a detour through float32 would drop 2^-30 and give 1)
    # 2^-133 is the smallest bf16 subnormal; 2^-140 is below half of it -> 0
    # 3.4e38 exceeds the largest bf16 value plus half an ulp -> inf
    vals = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-8 + 2**-30, -2.5, 0.0,
                     2.0**-133, 3 * 2.0**-134, 2.0**-140, 3.4e38, -3.4e38])
    want = np.array([1.0, 1.0, 1 + 2**-6, 1 + 2**-7, -2.5, 0.0,
                     2.0**-133, 2.0**-132, 0.0, np.inf, -np.inf])
    np.testing.assert_array_equal(oracle.round_to(vals, "bf16"), want)


def test_round_matches_torch_conversion():
    """For values exactly representable in float32, float32 -> bfloat16 in
    torch (round to nearest even) is an independent routine for the same
    rounding; float64 -> float32 is the C conversion."""
    rng = np.random.default_rng(8)
    v32 = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ref = torch.from_numpy(v32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_to(v32.astype(np.float64), "bf16"), ref)
    v64 = rng.standard_normal(1000) * 1e3
    np.testing.assert_array_equal(oracle.round_to(v64, "f32"), v64.astype(np.float32).astype(np.float64))


def test_rel_err():
    assert oracle.rel_err([1.0, 2.0], [1.0, 2.0]) == 0.0
    assert oracle.rel_err([1.0, 2.1], [1.0, 2.0]) == pytest.approx(0.05)
    assert oracle.rel_err([np.nan, 1.0], [1.0, 1.0]) == float("inf")
