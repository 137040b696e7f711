"""The PyTorch adapter (paper_2404_12406_amd.autograd): every layer under
every combination of requires_grad flags against the oracle, a converted
nn.Sequential end to end, and the synthetic deep CNN of Sec. 2.1 (Fig. 1):
after the forward pass the allocator holds exactly the inputs the save rule
keeps (closed form), where stock layers keep every input from the first
differentiable layer on."""
import itertools

import numpy as np
import pytest
import torch
from torch import nn

import oracle
import paper_2404_12406_amd as ms
from paper_2404_12406_amd import autograd as msa
import synth

from _gpu import TOL, dev, host

pytestmark = pytest.mark.gpu


def _leaf(a, dtype, rg):
    t = dev(a, dtype)
    t.requires_grad_(rg)
    return t


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("flags", list(itertools.product([False, True], repeat=3)))
def test_conv2d_function_masks(dtype, flags):
    rx, rw, rb = flags
    xs, ws = (2, 8, 9, 7), (16, 8, 3, 3)
    x = synth.normal(xs, 9800, dtype=dtype)
    w = synth.kaiming_uniform(ws, 9801, 72, dtype=dtype)
    b = synth.normal((16,), 9802, 0.1, dtype=dtype)
    xt, wt, bt = _leaf(x, dtype, rx), nn.Parameter(dev(w, dtype), requires_grad=rw), nn.Parameter(dev(b, dtype), requires_grad=rb)
    m = msa.MSConv2d(wt, bt, stride=(2, 1), padding=(1, 1))
    y = m(xt)
    assert oracle.rel_err(host(y), oracle.conv2d_forward(x, w, b, (2, 1), (1, 1))) <= TOL[dtype]
    if not (rx or rw or rb):
        assert y.grad_fn is None
        return
    gy = synth.normal(tuple(y.shape), 9803, dtype=dtype)
    y.backward(dev(gy, dtype))
    if rx:
        assert oracle.rel_err(host(xt.grad), oracle.conv2d_input_grad(gy, w, xs, (2, 1), (1, 1))) <= TOL[dtype]
    if rw:
        assert oracle.rel_err(host(m.weight.grad), oracle.conv2d_weight_grad(gy, x, ws, (2, 1), (1, 1))) <= TOL[dtype]
    if rb:
        assert oracle.rel_err(host(m.bias.grad), oracle.conv2d_bias_grad(gy)) <= TOL[dtype]
    assert (xt.grad is None) == (not rx) and (m.weight.grad is None) == (not rw) and (m.bias.grad is None) == (not rb)


@pytest.mark.parametrize("flags", list(itertools.product([False, True], repeat=3)))
def test_linear_and_bn_functions_masks(flags):
    rx, rw, rb = flags
    X = synth.normal((3, 5, 24), 9810, dtype="bf16")
    W = synth.normal((40, 24), 9811, 0.1, dtype="bf16")
    B = synth.normal((40,), 9812, 0.1, dtype="bf16")
    Xt = _leaf(X, "bf16", rx)
    lin = msa.MSLinear(nn.Parameter(dev(W, "bf16"), requires_grad=rw), nn.Parameter(dev(B, "bf16"), requires_grad=rb))
    Y = lin(Xt)
    assert tuple(Y.shape) == (3, 5, 40)
    X2 = X.reshape(15, 24)
    assert oracle.rel_err(host(Y).reshape(15, 40), oracle.linear_forward(X2, W, B)) <= TOL["bf16"]
    if rx or rw or rb:
        gY = synth.normal((3, 5, 40), 9813, dtype="bf16")
        Y.backward(dev(gY, "bf16"))
        g2 = gY.reshape(15, 40)
        if rx:
            assert oracle.rel_err(host(Xt.grad).reshape(15, 24), oracle.linear_input_grad(g2, W)) <= TOL["bf16"]
        if rw:
            assert oracle.rel_err(host(lin.weight.grad), oracle.linear_weight_grad(g2, X2)) <= TOL["bf16"]
        if rb:
            assert oracle.rel_err(host(lin.bias.grad), oracle.linear_bias_grad(g2)) <= TOL["bf16"]
    # BN-eval with gamma / beta flags
    x = synth.normal((2, 16, 5, 6), 9814, dtype="f32")
    mu, var = synth.normal((16,), 9815, 0.1), synth.uniform((16,), 9816, 0.5, 1.5)
    g, be = synth.uniform((16,), 9817, 0.5, 1.5), synth.normal((16,), 9818, 0.1)
    xt = _leaf(x, "f32", rx)
    bn = msa.MSBatchNorm2dEval(nn.Parameter(dev(g, "f32"), requires_grad=rw), nn.Parameter(dev(be, "f32"), requires_grad=rb),
                               dev(mu, "f32"), dev(var, "f32"), 1e-5)
    y = bn(xt)
    assert oracle.rel_err(host(y), oracle.bn_eval_forward(x, mu, var, g, be, 1e-5)) <= TOL["f32"]
    if rx or rw or rb:
        gy = synth.normal(x.shape, 9819)
        y.backward(dev(gy, "f32"))
        rdx, rdg, rdb = oracle.bn_eval_backward(gy, x, mu, var, g, 1e-5)
        if rx:
            assert oracle.rel_err(host(xt.grad), rdx) <= TOL["f32"]
        if rw:
            assert oracle.rel_err(host(bn.weight.grad), rdg) <= TOL["f32"]
        if rb:
            assert oracle.rel_err(host(bn.bias.grad), rdb) <= TOL["f32"]


def test_converted_sequential_end_to_end():
    """conv -> BN(eval) -> ReLU -> conv -> flatten -> linear, converted from
    torch.nn; gradients of the input and of the trainable parameters (the
    first conv frozen) against the oracle composed layer by layer in fp32."""
    torch.manual_seed(0)
    net = nn.Sequential(nn.Conv2d(8, 16, 3, padding=1), nn.BatchNorm2d(16), nn.ReLU(),
                        nn.Conv2d(16, 8, 3, stride=2, padding=1), nn.Flatten(), nn.Linear(8 * 4 * 5, 10)).cuda()
    with torch.no_grad():
        net[1].running_mean.normal_(0, 0.1)
        net[1].running_var.uniform_(0.5, 1.5)
    net.eval()
    net[0].weight.requires_grad_(False)
    net[0].bias.requires_grad_(False)
    params = {k: v.detach().cpu().numpy().astype(np.float64) for k, v in net.state_dict().items()}
    msa.convert(net)
    assert isinstance(net[0], msa.MSConv2d) and isinstance(net[1], msa.MSBatchNorm2dEval)
    assert isinstance(net[2], msa.MSReLU) and isinstance(net[5], msa.MSLinear)
    x = synth.normal((2, 8, 8, 9), 9820)
    xt = _leaf(x, "f32", True)
    y = net(xt)
    gy = synth.normal((2, 10), 9821)
    y.backward(dev(gy, "f32"))
    # oracle: forward
    h0 = oracle.conv2d_forward(x, params["0.weight"], params["0.bias"], (1, 1), (1, 1))
    h1 = oracle.bn_eval_forward(h0, params["1.running_mean"], params["1.running_var"], params["1.weight"],
                                params["1.bias"], 1e-5)
    h2 = oracle.relu_forward(h1)
    h3 = oracle.conv2d_forward(h2, params["3.weight"], params["3.bias"], (2, 2), (1, 1))
    f = h3.reshape(2, -1)
    out = oracle.linear_forward(f, params["5.weight"], params["5.bias"])
    assert oracle.rel_err(host(y), out) <= TOL["f32"]
    # oracle: backward
    g_f = oracle.linear_input_grad(gy, params["5.weight"])
    g3 = g_f.reshape(h3.shape)
    g2 = oracle.conv2d_input_grad(g3, params["3.weight"], h2.shape, (2, 2), (1, 1))
    g1 = oracle.relu_backward(g2, h1)
    g0 = oracle.bn_eval_backward(g1, h0, params["1.running_mean"], params["1.running_var"], params["1.weight"], 1e-5)[0]
    gx = oracle.conv2d_input_grad(g0, params["0.weight"], x.shape, (1, 1), (1, 1))
    assert oracle.rel_err(host(xt.grad), gx) <= TOL["f32"]
    assert oracle.rel_err(host(net[5].weight.grad), oracle.linear_weight_grad(gy, f)) <= TOL["f32"]
    assert oracle.rel_err(host(net[3].weight.grad), oracle.conv2d_weight_grad(g3, h2, params["3.weight"].shape, (2, 2), (1, 1))) <= TOL["f32"]
    assert net[0].weight.grad is None


@pytest.mark.parametrize("case", ["all", "layers_4_plus", "layer_4_only"])
def test_synthetic_deep_cnn_retains_exactly_the_saved_inputs(case):
    """Sec. 2.1 / Fig. 1 at test size: a stack of 8 bias-free 3x3 convs with
    8 channels, fp32; x = [4, 8, 64, 64] (512 KiB per layer input).  After
    the forward pass the allocator holds the final output plus the inputs the
    save rule keeps: 8 / 5 / 1 of them (stock layers: 8 / 5 / 5)."""
    from oracle import policy as P
    depth, xs = 8, (4, 8, 64, 64)
    nbytes = int(np.prod(xs)) * 4
    torch.manual_seed(1)
    convs = [nn.Conv2d(8, 8, 3, padding=1, bias=False).cuda() for _ in range(depth)]
    for i, c in enumerate(convs):
        layer = i + 1
        rw = case == "all" or (case == "layers_4_plus" and layer >= 4) or (case == "layer_4_only" and layer == 4)
        c.weight.requires_grad_(rw)
    net = msa.convert(nn.Sequential(*convs))
    x = torch.randn(xs, device="cuda").contiguous(memory_format=torch.channels_last)
    x.requires_grad_(case == "all")
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    y = net(x)
    torch.cuda.synchronize()
    held = torch.cuda.memory_allocated() - base - y.numel() * 4
    flags = [2 if c.weight.requires_grad else 0 for c in convs]
    masks = P.propagate(flags, case == "all")
    want = P.stack_saved_bytes([("conv2d", m, int(np.prod(xs)), "f32", True, False) for m in masks])
    stock = P.stack_saved_bytes([("conv2d", m, int(np.prod(xs)), "f32", True, False) for m in masks], P.PYTORCH_DEFAULT)
    kept = {"all": 8, "layers_4_plus": 5, "layer_4_only": 1}[case]
    assert want == kept * nbytes
    assert stock == {"all": 8, "layers_4_plus": 5, "layer_4_only": 5}[case] * nbytes
    # the input itself (held by the caller) is not counted: in case "all"
    # the first record borrows x, which `base` already includes
    assert held == want - (nbytes if case == "all" else 0)
    y.backward(torch.ones_like(y))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("flags", list(itertools.product([False, True], repeat=3)))
def test_conv_transpose2d_function_masks(dtype, flags):
    rx, rw, rb = flags
    xs, ws, st, pd, op = (2, 16, 5, 6), (16, 8, 4, 3), (2, 2), (1, 1), (1, 0)
    x = synth.normal(xs, 9830, dtype=dtype)
    w = synth.kaiming_uniform(ws, 9831, 8 * 12, dtype=dtype)
    b = synth.normal((8,), 9832, 0.1, dtype=dtype)
    xt = _leaf(x, dtype, rx)
    m = msa.MSConvTranspose2d(nn.Parameter(dev(w, dtype), requires_grad=rw),
                              nn.Parameter(dev(b, dtype), requires_grad=rb), st, pd, op)
    y = m(xt)
    assert oracle.rel_err(host(y), oracle.convt2d_forward(x, w, b, st, pd, op)) <= TOL[dtype]
    if not (rx or rw or rb):
        assert y.grad_fn is None
        return
    gy = synth.normal(tuple(y.shape), 9833, dtype=dtype)
    y.backward(dev(gy, dtype))
    if rx:
        assert oracle.rel_err(host(xt.grad), oracle.convt2d_input_grad(gy, w, xs, st, pd, op)) <= TOL[dtype]
    if rw:
        assert oracle.rel_err(host(m.weight.grad), oracle.convt2d_weight_grad(gy, x, ws, st, pd, op)) <= TOL[dtype]
    if rb:
        assert oracle.rel_err(host(m.bias.grad), oracle.convt2d_bias_grad(gy)) <= TOL[dtype]
    assert (xt.grad is None) == (not rx) and (m.weight.grad is None) == (not rw) and (m.bias.grad is None) == (not rb)


@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("flags", [(True, True, True), (True, False, False), (False, True, True)])
def test_one_dimensional_layers(transposed, flags):
    """Conv1d / ConvTranspose1d from torch.nn, converted, against the oracle
    of the 2-D layer with H = R = 1 (a plain [N, C, L] input that is not
    channels-inner is converted on the way in)."""
    rx, rw, rb = flags
    torch.manual_seed(3)
    if transposed:
        ref = nn.ConvTranspose1d(8, 16, 4, stride=2, padding=1, output_padding=1).cuda()
    else:
        ref = nn.Conv1d(8, 16, 3, stride=2, padding=1).cuda()
    w = ref.weight.detach().cpu().numpy().astype(np.float64)
    b = ref.bias.detach().cpu().numpy().astype(np.float64)
    ref.weight.requires_grad_(rw)
    ref.bias.requires_grad_(rb)
    net = msa.convert(nn.Sequential(ref))
    assert isinstance(net[0], msa.MSConvTranspose1d if transposed else msa.MSConv1d)
    x = synth.normal((3, 8, 21), 9840)
    xt = torch.from_numpy(x.astype(np.float32)).cuda().requires_grad_(rx)
    y = net(xt)
    x4, w4 = x[:, :, None, :], w[:, :, None, :]
    if transposed:
        want = oracle.convt2d_forward(x4, w4, b, (1, 2), (0, 1), (0, 1))[:, :, 0, :]
    else:
        want = oracle.conv2d_forward(x4, w4, b, (1, 2), (0, 1))[:, :, 0, :]
    assert tuple(y.shape) == want.shape
    assert oracle.rel_err(host(y), want) <= TOL["f32"]
    gy = synth.normal(want.shape, 9841)
    y.backward(torch.from_numpy(gy.astype(np.float32)).cuda())
    g4 = gy[:, :, None, :]
    if transposed:
        gx = oracle.convt2d_input_grad(g4, w4, x4.shape, (1, 2), (0, 1), (0, 1))
        gw = oracle.convt2d_weight_grad(g4, x4, w4.shape, (1, 2), (0, 1), (0, 1))
    else:
        gx = oracle.conv2d_input_grad(g4, w4, x4.shape, (1, 2), (0, 1))
        gw = oracle.conv2d_weight_grad(g4, x4, w4.shape, (1, 2), (0, 1))
    if rx:
        assert oracle.rel_err(host(xt.grad), gx[:, :, 0, :]) <= TOL["f32"]
    if rw:
        assert oracle.rel_err(host(net[0].weight.grad), gw[:, :, 0, :]) <= TOL["f32"]
    if rb:
        assert oracle.rel_err(host(net[0].bias.grad), oracle.conv2d_bias_grad(g4)) <= TOL["f32"]
    assert (net[0].weight.grad is None) == (not rw)


@pytest.mark.parametrize("kind", ["conv_transpose2d", "conv1d", "conv_transpose1d"])
@pytest.mark.parametrize("case", ["all", "layers_4_plus", "layer_4_only"])
def test_appendix_b_layers_retain_exactly_the_saved_inputs(kind, case):
    """App. B repeats the Fig. 1 experiment with the other layers that are
    linear in input and weight; at test size, a stack of 8 size-preserving
    layers with 8 channels and kernel 3, fp32: after the forward pass the
    allocator holds exactly the inputs the save rule keeps."""
    from oracle import policy as P
    depth = 8
    xs = (4, 8, 64, 64) if kind == "conv_transpose2d" else (16, 8, 1024)
    nel = int(np.prod(xs))
    torch.manual_seed(2)
    mk = {"conv_transpose2d": lambda: nn.ConvTranspose2d(8, 8, 3, padding=1, bias=False),
          "conv1d": lambda: nn.Conv1d(8, 8, 3, padding=1, bias=False),
          "conv_transpose1d": lambda: nn.ConvTranspose1d(8, 8, 3, padding=1, bias=False)}[kind]
    layers = [mk().cuda() for _ in range(depth)]
    for i, c in enumerate(layers):
        layer = i + 1
        c.weight.requires_grad_(case == "all" or (case == "layers_4_plus" and layer >= 4)
                                or (case == "layer_4_only" and layer == 4))
    net = msa.convert(nn.Sequential(*layers))
    x = torch.randn(xs, device="cuda")
    x = x.contiguous(memory_format=torch.channels_last) if len(xs) == 4 else x.transpose(1, 2).contiguous().transpose(1, 2)
    x.requires_grad_(case == "all")
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    y = net(x)
    torch.cuda.synchronize()
    held = torch.cuda.memory_allocated() - base - y.numel() * 4
    kind2 = "conv2d" if kind == "conv1d" else "conv_transpose2d"
    masks = P.propagate([2 if c.weight.requires_grad else 0 for c in layers], case == "all")
    want = P.stack_saved_bytes([(kind2, m, nel, "f32", True, False) for m in masks])
    assert want == {"all": 8, "layers_4_plus": 5, "layer_4_only": 1}[case] * nel * 4
    assert held == want - (nel * 4 if case == "all" else 0)
    y.backward(torch.ones_like(y))
    assert (layers[3].weight.grad is not None) and (layers[0].weight.grad is None) == (case != "all")


def test_inplace_change_of_a_borrowed_input_is_refused():
    """A conv whose weight trains borrows its input; writing that input in
    place before backward would give a wrong weight gradient, so backward
    raises (as stock autograd does for its saved tensors).  An input the
    record does not borrow (frozen weight) may be changed freely."""
    from paper_2404_12406_amd import autograd as msa
    torch.manual_seed(0)
    conv = msa.convert(torch.nn.Sequential(torch.nn.Conv2d(8, 16, 3, padding=1))).cuda()
    x = torch.randn(2, 8, 6, 6, device="cuda")
    y = conv(x)
    x.add_(1.0)
    with pytest.raises(RuntimeError, match="inplace"):
        y.sum().backward()
    conv[0].weight.requires_grad_(False)
    xi = torch.randn(2, 8, 6, 6, device="cuda", requires_grad=True)
    xx = xi * 1.0
    y = conv(xx)
    xx.add_(1.0)                      # not borrowed: the input gradient needs W only
    y.sum().backward()
    assert xi.grad is not None
