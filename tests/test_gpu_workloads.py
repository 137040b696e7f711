"""GPU parity of the five synthetic workloads against the oracle.

* Reduced sizes (ragged tails, several tiles): every element of every
  output and requested gradient of a whole stack, plus the ledger's peak of
  retained bytes against the closed form.
* Full sizes, in the launch configuration the benchmark times: rows of a
  Linear stack and images of a conv stack are independent, so the oracle
  recomputes sampled rows / images end to end from the same seeded inputs;
  single layers are checked at sampled entries (including borders), and
  bias / BN reductions in full.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_12406_amd as ms
from oracle import policy as P
from synth import draw, gpu
from synth import workloads as wl

from _gpu import check, host

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ oracle of a chain
def oracle_chain(ca, dtype, rows=None, want_grads=True):
    """Forward (and masked backward) of a drawn chain with the oracle,
    optionally restricted to a subset of batch rows / images.  Activations
    and propagated gradients are rounded to the storage dtype where the GPU
    stores them."""
    x = ca.x if rows is None else ca.x[rows]
    acts = [x]
    for la in ca.layers:
        s = la.spec
        a = acts[-1]
        if s.kind == "conv2d":
            y = oracle.conv2d_forward(a, la.W, la.b, s.stride, s.pad)
        elif s.kind == "conv_transpose2d":
            y = oracle.convt2d_forward(a, la.W, la.b, s.stride, s.pad, s.out_pad)
        elif s.kind == "linear":
            y = oracle.linear_forward(a, la.W, la.b)
        elif s.kind == "bn_eval":
            y = oracle.bn_eval_forward(a, la.running_mean, la.running_var, la.W, la.b, s.eps)
        else:
            y = oracle.avgpool_forward(a)
        acts.append(oracle.round_to(y, dtype))
    if not want_grads:
        return acts, None
    g = ca.grad_y if rows is None else ca.grad_y[rows]
    grads = [None] * len(ca.layers)
    for i in range(len(ca.layers) - 1, -1, -1):
        la, s, a = ca.layers[i], ca.layers[i].spec, acts[i]
        m = s.mask
        if m == 0:
            break
        gx = gw = gb = None
        if s.kind == "conv2d":
            if m & 1:
                gx = oracle.conv2d_input_grad(g, la.W, a.shape, s.stride, s.pad)
            if m & 2:
                gw = oracle.conv2d_weight_grad(g, a, la.W.shape, s.stride, s.pad)
            if m & 4:
                gb = oracle.conv2d_bias_grad(g)
        elif s.kind == "conv_transpose2d":
            if m & 1:
                gx = oracle.convt2d_input_grad(g, la.W, a.shape, s.stride, s.pad, s.out_pad)
            if m & 2:
                gw = oracle.convt2d_weight_grad(g, a, la.W.shape, s.stride, s.pad, s.out_pad)
            if m & 4:
                gb = oracle.convt2d_bias_grad(g)
        elif s.kind == "linear":
            if m & 1:
                gx = oracle.linear_input_grad(g, la.W)
            if m & 2:
                gw = oracle.linear_weight_grad(g, a)
            if m & 4:
                gb = oracle.linear_bias_grad(g)
        elif s.kind == "bn_eval":
            gx, gw, gb = oracle.bn_eval_backward(g, a, la.running_mean, la.running_var, la.W, s.eps,
                                                 bool(m & 1), bool(m & 2), bool(m & 4))
        else:
            gx = oracle.avgpool_backward(g, a.shape)
        grads[i] = (gx, gw, gb)
        if gx is None:
            break
        g = oracle.round_to(gx, dtype)
    return acts, grads


def run_gpu_chain(ca, dtype):
    chain = gpu.build_chain(ca, dtype)
    live0, _ = ms.ledger_read()
    ms.ledger_reset()
    chain.forward()
    torch.cuda.synchronize()
    _, peak = ms.ledger_read()
    chain.backward()
    torch.cuda.synchronize()
    return chain, peak - live0


def _layers_bytes(w):
    return [(l.kind, l.mask, int(np.prod(l.in_shape)), w.dtype, l.kind != "avgpool", l.has_bias) for l in w.layers]


def pick_rows(t, rows):
    """Device tensor -> float64 host array, restricted to batch `rows`."""
    if rows is None:
        return host(t)
    return host(t[torch.as_tensor(rows, device=t.device)])


def compare_chain(chain, acts, grads, dtype, rows=None, tol=None):
    for i, a in enumerate(acts[1:]):
        check(f"act{i}", pick_rows(chain.acts[i + 1], rows), a, dtype, tol)
    if grads is None:
        return
    for i, g in enumerate(grads):
        if g is None:
            continue
        gx, gw, gb = chain.grads[i]
        if g[0] is not None:
            check(f"gx{i}", pick_rows(gx, rows), g[0], dtype, tol)
        if rows is None:
            if g[1] is not None:
                check(f"gW{i}", host(gw), g[1], dtype, tol)
            if g[2] is not None:
                check(f"gb{i}", host(gb), g[2], dtype, tol)


# ------------------------------------------------------------------ reduced-size stacks
@pytest.mark.parametrize("variant", [False, True])
def test_resnet18_shaped_stack_reduced(variant):
    w = wl.resnet18_shaped_bf16(batch=2, image=72, input_requires_grad=variant)
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "bf16")
    acts, grads = oracle_chain(ca, "bf16")
    compare_chain(chain, acts, grads, "bf16")
    assert peak == P.stack_saved_bytes(_layers_bytes(w), P.SELECTIVE)


def test_linear_stack_reduced():
    w = wl.linear_stack_bf16(m=300)
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "bf16")
    acts, grads = oracle_chain(ca, "bf16")
    compare_chain(chain, acts, grads, "bf16")
    assert peak == 0
    assert P.stack_saved_bytes(_layers_bytes(w), P.ALL_TRUE) == 300 * (1024 + 4096 + 1024 + 4096) * 2


def test_encoder_linears_reduced():
    w = wl.encoder_linears_bf16(layers=1, tokens=200)
    for ca in draw.chains(w):
        chain, peak = run_gpu_chain(ca, "bf16")
        acts, grads = oracle_chain(ca, "bf16")
        compare_chain(chain, acts, grads, "bf16")
        assert peak == 0


def test_single_conv_f32_workload():
    w = wl.single_conv_f32()
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "f32")
    acts, grads = oracle_chain(ca, "f32")
    compare_chain(chain, acts, grads, "f32")
    assert peak == 0
    assert P.stack_saved_bytes(_layers_bytes(w), P.PYTORCH_DEFAULT) == 524288


# ------------------------------------------------------------------ full sizes
def _sample_rows(n, k, seed):
    rng = np.random.default_rng(seed)
    rows = set([0, n - 1]) | set(rng.choice(n, size=min(k, n), replace=False).tolist())
    return np.array(sorted(rows))


def test_linear_stack_full_size_rows():
    """The headline workload at full size: 64 sampled rows through the whole
    stack forward and backward, the last bias gradient in full and the
    earlier ones through db_l = db_{l+1} W_{l+1} (linearity)."""
    w = wl.linear_stack_bf16()
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "bf16")
    assert peak == 0
    rows = _sample_rows(4096, 62, 1)
    acts, grads = oracle_chain(ca, "bf16", rows=rows)
    compare_chain(chain, acts, grads, "bf16", rows=rows)
    db_last = oracle.linear_bias_grad(ca.grad_y)
    check("db3", host(chain.grads[3][2]), db_last, "bf16")
    ref = db_last
    for l in (2, 1, 0):
        ref = oracle.linear_input_grad(ref[None, :], ca.layers[l + 1].W)[0]
        check(f"db{l}", host(chain.grads[l][2]), ref, "bf16")


def test_encoder_linears_full_size_rows():
    w = wl.encoder_linears_bf16(layers=1)          # the four linear shapes at M = 16*512
    rows = _sample_rows(8192, 30, 2)
    for ci, ca in enumerate(draw.chains(w)):
        chain, peak = run_gpu_chain(ca, "bf16")
        assert peak == 0
        acts, grads = oracle_chain(ca, "bf16", rows=rows)
        compare_chain(chain, acts, grads, "bf16", rows=rows)
        del chain
        torch.cuda.empty_cache()


@pytest.mark.parametrize("variant", [False, True])
def test_resnet18_shaped_full_size_one_image(variant):
    """Full batch of 64 at 224x224 on the GPU; the oracle recomputes image 37
    through the whole stack (and, in the input variant, back to the image)."""
    w = wl.resnet18_shaped_bf16(input_requires_grad=variant)
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "bf16")
    assert peak == P.stack_saved_bytes(_layers_bytes(w), P.SELECTIVE)
    rows = np.array([37])
    acts, grads = oracle_chain(ca, "bf16", rows=rows, want_grads=variant)
    compare_chain(chain, acts, grads, "bf16", rows=rows)
    del chain
    torch.cuda.empty_cache()


def _conv_layer_full(spec, dtype, seed, samples=2048):
    la = draw.layer_arrays(spec, dtype)
    import synth
    x = synth.normal(spec.in_shape, seed, dtype=dtype)
    gy = synth.normal(spec.out_shape(), seed + 1, dtype=dtype)
    W = gpu.dev(la.W, dtype)
    B = gpu.dev(la.b, dtype)
    y, rec = ms.layer_forward(ms.Conv2d(spec.stride, spec.pad), gpu.dev(x, dtype), W, B, spec.mask)
    yh = host(y)
    rng = np.random.default_rng(seed)
    N, K, Pp, Q = yh.shape
    idx = np.stack([rng.integers(0, d, samples) for d in (N, K, Pp, Q)], 1)
    idx = np.concatenate([idx, [[0, 0, 0, 0], [N - 1, K - 1, Pp - 1, Q - 1], [0, K - 1, 0, Q - 1],
                                [N - 1, 0, Pp - 1, 0]]])
    ref = oracle.conv2d_forward_at(x, la.W, la.b, spec.stride, spec.pad, idx)
    check("y@", yh[tuple(idx.T)], ref, dtype)
    if rec is None:
        return
    gx, gw, gb = ms.layer_backward(rec, gpu.dev(gy, dtype))
    if gx is not None:
        gxh = host(gx)
        Nn, C, H, Wd = gxh.shape
        idx = np.stack([rng.integers(0, d, samples) for d in (Nn, C, H, Wd)], 1)
        idx = np.concatenate([idx, [[0, 0, 0, 0], [Nn - 1, C - 1, H - 1, Wd - 1], [0, 0, H - 1, 0]]])
        ref = oracle.conv2d_input_grad_at(gy, la.W, spec.in_shape, spec.stride, spec.pad, idx)
        check("dx@", gxh[tuple(idx.T)], ref, dtype)
    if gw is not None:
        gwh = host(gw)
        idx = np.stack([rng.integers(0, d, 512) for d in gwh.shape], 1)
        idx = np.concatenate([idx, [[0, 0, 0, 0], [d - 1 for d in gwh.shape]]])
        ref = oracle.conv2d_weight_grad_at(gy, x, la.W.shape, spec.stride, spec.pad, idx)
        check("dW@", gwh[tuple(idx.T)], ref, dtype)
    if gb is not None:
        check("db", host(gb), oracle.conv2d_bias_grad(gy), dtype)


@pytest.mark.parametrize("mk", ["00", "10", "01", "11"])
@pytest.mark.parametrize("pointwise", [False, True])
def test_conv_sweep_full_size(mk, pointwise):
    w = wl.conv_sweep_bf16(mk, pointwise=pointwise)
    _conv_layer_full(w.layers[0], "bf16", 4100 + 10 * int(pointwise))


def test_resnet18_shaped_layers_full_size():
    """Every conv of the stack at its full size, with both masks it meets
    (frozen forward, and input-gradient for the input variant)."""
    w = wl.resnet18_shaped_bf16(input_requires_grad=True)
    for i, spec in enumerate(w.layers):
        if spec.kind == "conv2d":
            _conv_layer_full(spec, "bf16", 4200 + i, samples=1024)
            torch.cuda.empty_cache()


def test_resnet18_shaped_bn_and_head_full_size():
    import synth
    w = wl.resnet18_shaped_bf16(input_requires_grad=True)
    for i, spec in enumerate(w.layers):
        if spec.kind not in ("bn_eval", "linear"):
            continue
        if spec.kind == "bn_eval" and spec.in_shape[1] not in (64, 512):
            continue   # stem-sized and last-stage BN cover both ends of the channel range
        la = draw.layer_arrays(spec, "bf16")
        x = synth.normal(spec.in_shape, 4300 + i, dtype="bf16")
        gy = synth.normal(spec.out_shape(), 4400 + i, dtype="bf16")
        if spec.kind == "bn_eval":
            bn = ms.BatchNormEval(gpu.dev(la.running_mean, "bf16"), gpu.dev(la.running_var, "bf16"), spec.eps)
            y, rec = ms.layer_forward(bn, gpu.dev(x, "bf16"), gpu.dev(la.W, "bf16"), gpu.dev(la.b, "bf16"), 7)
            check("bn y", host(y), oracle.bn_eval_forward(x, la.running_mean, la.running_var, la.W, la.b), "bf16")
            gx, gg, gb = ms.layer_backward(rec, gpu.dev(gy, "bf16"))
            rx, rg, rb = oracle.bn_eval_backward(gy, x, la.running_mean, la.running_var, la.W)
            check("bn dx", host(gx), rx, "bf16")
            check("bn dgamma", host(gg), rg, "bf16")
            check("bn dbeta", host(gb), rb, "bf16")
        else:
            y, rec = ms.layer_forward(ms.Linear(), gpu.dev(x, "bf16"), gpu.dev(la.W, "bf16"), gpu.dev(la.b, "bf16"), 6)
            check("fc y", host(y), oracle.linear_forward(x, la.W, la.b), "bf16")
            assert rec.account()["saved_activation_bytes"] == 65536
            _, gw, gb = ms.layer_backward(rec, gpu.dev(gy, "bf16"))
            check("fc dW", host(gw), oracle.linear_weight_grad(gy, x), "bf16")
            check("fc db", host(gb), oracle.linear_bias_grad(gy), "bf16")
        torch.cuda.empty_cache()


# ------------------------------------------------------------------ transposed convolutions
def test_decoder_convt_stack_reduced():
    """The three-layer ConvTranspose2d decoder at batch 2, every element of
    every activation and gradient, and the ledger against the closed form."""
    w = wl.decoder_convt_bf16(batch=2)
    ca = draw.chains(w)[0]
    chain, peak = run_gpu_chain(ca, "bf16")
    acts, grads = oracle_chain(ca, "bf16")
    compare_chain(chain, acts, grads, "bf16")
    assert peak == P.stack_saved_bytes(_layers_bytes(w), P.SELECTIVE)


def _convt_layer_full(spec, dtype, seed, samples=2048):
    import synth
    la = draw.layer_arrays(spec, dtype)
    x = synth.normal(spec.in_shape, seed, dtype=dtype)
    gy = synth.normal(spec.out_shape(), seed + 1, dtype=dtype)
    st, pd, op = spec.stride, spec.pad, spec.out_pad
    y, rec = ms.layer_forward(ms.ConvTranspose2d(st, pd, op), gpu.dev(x, dtype), gpu.dev(la.W, dtype),
                              gpu.dev(la.b, dtype), spec.mask)
    yh = host(y)
    rng = np.random.default_rng(seed)
    dims = yh.shape
    idx = np.stack([rng.integers(0, d, samples) for d in dims], 1)
    idx = np.concatenate([idx, [[0, 0, 0, 0], [d - 1 for d in dims], [0, dims[1] - 1, 0, dims[3] - 1],
                                [dims[0] - 1, 0, dims[2] - 1, 0]]])
    check("y@", yh[tuple(idx.T)], oracle.convt2d_forward_at(x, la.W, la.b, st, pd, op, idx), dtype)
    if rec is None:
        return
    gx, gw, gb = ms.layer_backward(rec, gpu.dev(gy, dtype))
    if gx is not None:
        gxh = host(gx)
        idx = np.stack([rng.integers(0, d, samples) for d in gxh.shape], 1)
        idx = np.concatenate([idx, [[0, 0, 0, 0], [d - 1 for d in gxh.shape]]])
        check("dx@", gxh[tuple(idx.T)], oracle.convt2d_input_grad_at(gy, la.W, spec.in_shape, st, pd, op, idx),
              dtype)
    if gw is not None:
        gwh = host(gw)
        idx = np.stack([rng.integers(0, d, 512) for d in gwh.shape], 1)
        idx = np.concatenate([idx, [[0, 0, 0, 0], [d - 1 for d in gwh.shape]]])
        check("dW@", gwh[tuple(idx.T)], oracle.convt2d_weight_grad_at(gy, x, la.W.shape, st, pd, op, idx), dtype)
    if gb is not None:
        check("db", host(gb), oracle.convt2d_bias_grad(gy), dtype)


def test_decoder_convt_layers_full_size():
    """Every layer of the decoder at the benchmark's batch of 32, with every
    gradient requested, at sampled entries (corners included); the bias
    gradient in full."""
    w = wl.decoder_convt_bf16()
    for i, spec in enumerate(w.layers):
        _convt_layer_full(spec, "bf16", 4600 + 10 * i)
        torch.cuda.empty_cache()
