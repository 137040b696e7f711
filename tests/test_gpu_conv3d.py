"""GPU parity of Conv3d and ConvTranspose3d (App. B) against the oracle for
every mask, in fp32 and bf16: depth strides and pads, output padding,
folded channel counts T*C that are and are not multiples of 8, and the
converted torch.nn layers with the Fig. 1 / App. B retained-bytes result."""
import itertools

import numpy as np
import pytest
import torch
from torch import nn

import oracle
import paper_2404_12406_amd as ms
from paper_2404_12406_amd import autograd as msa
import synth
from oracle import policy as P

from _gpu import TOL, TORCH_DT, check, host

pytestmark = pytest.mark.gpu


def dev5(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_DT[dtype])
    if t.dim() == 5:
        t = t.contiguous(memory_format=torch.channels_last_3d)
    return t.cuda()


CASES = [
    # x shape, C_out, (T, R, S), stride, pad, out_pad (None: Conv3d), dtype
    ((2, 8, 6, 7, 5), 16, (3, 3, 3), (1, 1, 1), (1, 1, 1), None, "bf16"),
    ((1, 3, 5, 9, 8), 8, (3, 1, 2), (2, 1, 2), (1, 0, 1), None, "bf16"),      # T*C = 9: padded channels
    ((2, 16, 4, 5, 5), 24, (2, 3, 3), (2, 2, 1), (0, 1, 1), None, "bf16"),
    ((2, 4, 5, 6, 4), 6, (3, 3, 3), (1, 1, 1), (1, 1, 1), None, "f32"),
    ((2, 16, 3, 4, 4), 8, (2, 4, 4), (2, 2, 2), (0, 1, 1), (1, 0, 1), "bf16"),
    ((1, 8, 4, 5, 3), 3, (3, 3, 3), (1, 2, 1), (1, 1, 1), (0, 1, 0), "bf16"),  # 3 output channels
    ((2, 5, 3, 4, 4), 4, (3, 2, 3), (2, 1, 2), (1, 0, 1), (1, 0, 0), "f32"),
    ((1, 8, 2, 3, 3), 8, (1, 1, 1), (3, 2, 2), (0, 0, 0), (2, 1, 0), "bf16"),  # kernel < stride: holes
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("mask", range(8))
def test_conv3d_all_masks(case, mask):
    xs, co, k, st, pd, op, dt = CASES[case]
    tr = op is not None
    seed = 8200 + 10 * case
    ws = (xs[1], co) + k if tr else (co, xs[1]) + k
    x = synth.normal(xs, seed, dtype=dt)
    w = synth.kaiming_uniform(ws, seed + 1, ws[1] * k[0] * k[1] * k[2], dtype=dt)
    b = synth.normal((co,), seed + 2, 0.1, dtype=dt)
    if tr:
        spec = ms.ConvTranspose3d(st, pd, op)
        y_ref = oracle.convt3d_forward(x, w, b, st, pd, op)
    else:
        spec = ms.Conv3d(st, pd)
        y_ref = oracle.conv3d_forward(x, w, b, st, pd)
    y, rec = ms.layer_forward(spec, dev5(x, dt), dev5(w, dt), dev5(b, dt), mask)
    assert tuple(y.shape) == y_ref.shape
    check("y", host(y), y_ref, dt)
    if mask == 0:
        assert rec is None
        return
    kind = "conv_transpose3d" if tr else "conv3d"
    assert rec.account()["saved_activation_bytes"] == P.saved_activation_bytes(kind, mask, x.size, dt)
    gy = synth.normal(y_ref.shape, seed + 3, dtype=dt)
    gx, gw, gb = ms.layer_backward(rec, dev5(gy, dt))
    assert (gx is not None) == bool(mask & 1) and (gw is not None) == bool(mask & 2) and (gb is not None) == bool(mask & 4)
    if tr:
        if gx is not None:
            check("dx", host(gx), oracle.convt3d_input_grad(gy, w, xs, st, pd, op), dt)
        if gw is not None:
            check("dW", host(gw), oracle.convt3d_weight_grad(gy, x, ws, st, pd, op), dt)
    else:
        if gx is not None:
            check("dx", host(gx), oracle.conv3d_input_grad(gy, w, xs, st, pd), dt)
        if gw is not None:
            check("dW", host(gw), oracle.conv3d_weight_grad(gy, x, ws, st, pd), dt)
    if gb is not None:
        check("db", host(gb), oracle.bias_grad5(gy), dt)
    rec.free()


@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("flags", list(itertools.product([False, True], repeat=3)))
def test_converted_3d_layers(transposed, flags):
    rx, rw, rb = flags
    torch.manual_seed(11)
    ref = (nn.ConvTranspose3d(8, 16, 3, stride=(2, 1, 2), padding=1, output_padding=(1, 0, 0)) if transposed
           else nn.Conv3d(8, 16, 3, stride=(1, 2, 1), padding=(1, 0, 1))).cuda()
    w = ref.weight.detach().cpu().double().numpy()
    b = ref.bias.detach().cpu().double().numpy()
    ref.weight.requires_grad_(rw)
    ref.bias.requires_grad_(rb)
    net = msa.convert(nn.Sequential(ref))
    assert isinstance(net[0], msa.MSConvTranspose3d if transposed else msa.MSConv3d)
    x = synth.normal((2, 8, 4, 6, 5), 8300)
    xt = torch.from_numpy(x.astype(np.float32)).cuda().requires_grad_(rx)     # plain layout: converted on the way in
    y = net(xt)
    if transposed:
        want = oracle.convt3d_forward(x, w, b, (2, 1, 2), (1, 1, 1), (1, 0, 0))
    else:
        want = oracle.conv3d_forward(x, w, b, (1, 2, 1), (1, 0, 1))
    assert oracle.rel_err(host(y), want) <= TOL["f32"]
    if not (rx or rw or rb):
        assert y.grad_fn is None
        return
    gy = synth.normal(want.shape, 8301)
    y.backward(torch.from_numpy(gy.astype(np.float32)).cuda())
    if rx:
        gx = (oracle.convt3d_input_grad(gy, w, x.shape, (2, 1, 2), (1, 1, 1), (1, 0, 0)) if transposed
              else oracle.conv3d_input_grad(gy, w, x.shape, (1, 2, 1), (1, 0, 1)))
        assert oracle.rel_err(host(xt.grad), gx) <= TOL["f32"]
    if rw:
        gw = (oracle.convt3d_weight_grad(gy, x, w.shape, (2, 1, 2), (1, 1, 1), (1, 0, 0)) if transposed
              else oracle.conv3d_weight_grad(gy, x, w.shape, (1, 2, 1), (1, 0, 1)))
        assert oracle.rel_err(host(net[0].weight.grad), gw) <= TOL["f32"]
    if rb:
        assert oracle.rel_err(host(net[0].bias.grad), oracle.bias_grad5(gy)) <= TOL["f32"]
    assert (net[0].weight.grad is None) == (not rw)


@pytest.mark.parametrize("kind", ["conv3d", "conv_transpose3d"])
@pytest.mark.parametrize("case", ["all", "layers_4_plus", "layer_4_only"])
def test_appendix_b_3d_layers_retain_exactly_the_saved_inputs(kind, case):
    """App. B's 3-D probes at test size: 8 size-preserving layers with 8
    channels and kernel 3 on (2, 8, 16, 16, 16) fp32."""
    depth, xs = 8, (2, 8, 16, 16, 16)
    nel = int(np.prod(xs))
    torch.manual_seed(4)
    mk = (lambda: nn.Conv3d(8, 8, 3, padding=1, bias=False)) if kind == "conv3d" else \
         (lambda: nn.ConvTranspose3d(8, 8, 3, padding=1, bias=False))
    layers = [mk().cuda() for _ in range(depth)]
    for i, c in enumerate(layers):
        layer = i + 1
        c.weight.requires_grad_(case == "all" or (case == "layers_4_plus" and layer >= 4)
                                or (case == "layer_4_only" and layer == 4))
    net = msa.convert(nn.Sequential(*layers))
    x = torch.randn(xs, device="cuda").contiguous(memory_format=torch.channels_last_3d)
    x.requires_grad_(case == "all")
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    y = net(x)
    torch.cuda.synchronize()
    held = torch.cuda.memory_allocated() - base - y.numel() * 4
    masks = P.propagate([2 if c.weight.requires_grad else 0 for c in layers], case == "all")
    want = P.stack_saved_bytes([(kind, m, nel, "f32", True, False) for m in masks])
    assert want == {"all": 8, "layers_4_plus": 5, "layer_4_only": 1}[case] * nel * 4
    assert held == want - (nel * 4 if case == "all" else 0)
    y.backward(torch.ones_like(y))
