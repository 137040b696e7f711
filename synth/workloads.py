"""Shapes, masks, init laws and seeds of the five synthetic workloads.

A workload is a list of layer descriptions.  Nothing here computes a layer;
it only says what each layer is and how its inputs are drawn, so that the
oracle checks, the GPU tests and the benchmark all build the same tensors.

Mask bits: 1 = the layer input requires grad, 2 = the weight (BN: gamma)
requires grad, 4 = the bias (BN: beta) requires grad.

Seeds: tensor t of workload c is drawn with seed 1000*c + t, t counting the
tensors of every layer in order (x, W, b, grad_y, running_mean, running_var,
gamma, beta as present).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

MASK_INPUT, MASK_WEIGHT, MASK_BIAS = 1, 2, 4


@dataclass
class LayerSpec:
    kind: str                      # "conv2d" | "conv_transpose2d" | "linear" | "bn_eval" | "avgpool"
    name: str
    in_shape: Tuple[int, ...]      # conv/bn/avgpool: logical (N, C, H, W); linear: (M, K_in)
    out_ch: int = 0                # conv: K; transposed conv: C_out; linear: N_out
    ksize: Tuple[int, int] = (1, 1)
    stride: Tuple[int, int] = (1, 1)
    pad: Tuple[int, int] = (0, 0)
    out_pad: Tuple[int, int] = (0, 0)   # transposed conv only
    has_bias: bool = False
    mask: int = 0
    eps: float = 1e-5
    # init laws: name -> (law, params); law in {"normal", "uniform", "kaiming"}
    init: Dict[str, Tuple[str, tuple]] = field(default_factory=dict)
    seeds: Dict[str, int] = field(default_factory=dict)
    chained_input: bool = True     # input is the previous layer's output

    def out_shape(self) -> Tuple[int, ...]:
        if self.kind == "conv2d":
            n, _, h, w = self.in_shape
            r, s = self.ksize
            p = (h + 2 * self.pad[0] - r) // self.stride[0] + 1
            q = (w + 2 * self.pad[1] - s) // self.stride[1] + 1
            return (n, self.out_ch, p, q)
        if self.kind == "conv_transpose2d":
            n, _, h, w = self.in_shape
            r, s = self.ksize
            ho = (h - 1) * self.stride[0] - 2 * self.pad[0] + r + self.out_pad[0]
            wo = (w - 1) * self.stride[1] - 2 * self.pad[1] + s + self.out_pad[1]
            return (n, self.out_ch, ho, wo)
        if self.kind == "linear":
            return (self.in_shape[0], self.out_ch)
        if self.kind == "bn_eval":
            return tuple(self.in_shape)
        if self.kind == "avgpool":
            return (self.in_shape[0], self.in_shape[1])
        raise ValueError(self.kind)

    def weight_shape(self) -> Optional[Tuple[int, ...]]:
        if self.kind == "conv2d":
            return (self.out_ch, self.in_shape[1], self.ksize[0], self.ksize[1])
        if self.kind == "conv_transpose2d":
            return (self.in_shape[1], self.out_ch, self.ksize[0], self.ksize[1])
        if self.kind == "linear":
            return (self.out_ch, self.in_shape[1])
        if self.kind == "bn_eval":
            return (self.in_shape[1],)
        return None


@dataclass
class Workload:
    index: int                     # 1-based workload number
    name: str
    dtype: str                     # "f32" | "bf16"
    layers: List[LayerSpec]
    input_law: Tuple[str, tuple] = ("normal", (0.0, 1.0))
    grad_law: Tuple[str, tuple] = ("normal", (0.0, 1.0))
    input_seed: int = 0
    note: str = ""


class _Seeds:
    def __init__(self, cfg: int):
        self.base = 1000 * cfg
        self.t = 0

    def __call__(self) -> int:
        s = self.base + self.t
        self.t += 1
        return s


def _conv(name, in_shape, k, r, stride, pad, mask, seeds, bias, bias_law=None):
    c = in_shape[1]
    fan_in = c * r * r
    init = {"W": ("kaiming", (fan_in,))}
    sd = {"W": seeds()}
    if bias:
        init["b"] = bias_law or ("kaiming", (fan_in,))
        sd["b"] = seeds()
    return LayerSpec("conv2d", name, tuple(in_shape), out_ch=k, ksize=(r, r),
                     stride=(stride, stride), pad=(pad, pad), has_bias=bias,
                     mask=mask, init=init, seeds=sd)


def _convt(name, in_shape, c_out, r, stride, pad, mask, seeds, bias):
    """Transposed conv with PyTorch's default init law: the fan-in of a
    ConvTranspose weight [C_in, C_out, R, S] is C_out * R * S."""
    fan_in = c_out * r * r
    init = {"W": ("kaiming", (fan_in,))}
    sd = {"W": seeds()}
    if bias:
        init["b"] = ("kaiming", (fan_in,))
        sd["b"] = seeds()
    return LayerSpec("conv_transpose2d", name, tuple(in_shape), out_ch=c_out, ksize=(r, r),
                     stride=(stride, stride), pad=(pad, pad), has_bias=bias,
                     mask=mask, init=init, seeds=sd)


def _bn(name, in_shape, mask, seeds):
    init = {"running_mean": ("normal", (0.0, 0.1)),
            "running_var": ("uniform", (0.5, 1.5)),
            "W": ("uniform", (0.5, 1.5)),
            "b": ("normal", (0.0, 0.1))}
    sd = {k: seeds() for k in ("running_mean", "running_var", "W", "b")}
    return LayerSpec("bn_eval", name, tuple(in_shape), has_bias=True, mask=mask,
                     init=init, seeds=sd)


def _linear(name, m, k_in, n_out, mask, seeds, w_law, b_law, chained=True):
    init = {"W": w_law, "b": b_law}
    sd = {"W": seeds(), "b": seeds()}
    return LayerSpec("linear", name, (m, k_in), out_ch=n_out, has_bias=True,
                     mask=mask, init=init, seeds=sd, chained_input=chained)


def single_conv_f32() -> Workload:
    """Single 3x3 Conv2d in fp32, input-only mask."""
    s = _Seeds(1)
    x_seed = s()
    layer = _conv("conv", (8, 16, 32, 32), 32, 3, 1, 1, MASK_INPUT, s, bias=True,
                  bias_law=("normal", (0.0, 0.1)))
    w = Workload(1, "single_conv2d_f32", "f32", [layer], input_seed=x_seed,
                 note="x[8,16,32,32], W[32,16,3,3], s1 p1, mask (I)")
    w.grad_seed = s()
    return w


def linear_stack_bf16(m: int = 4096) -> Workload:
    """Four bf16 Linear layers 1024->4096->1024->4096->1024, weights frozen,
    biases trainable, input requires grad."""
    s = _Seeds(2)
    x_seed = s()
    dims = [1024, 4096, 1024, 4096, 1024]
    layers = []
    for i in range(4):
        layers.append(_linear(f"fc{i}", m, dims[i], dims[i + 1],
                              MASK_INPUT | MASK_BIAS, s,
                              ("normal", (0.0, 0.02)), ("normal", (0.0, 0.02))))
    w = Workload(2, "linear_stack_bf16", "bf16", layers, input_seed=x_seed,
                 note=f"X[{m},1024], 1024->4096->1024->4096->1024, mask (I,B)")
    w.grad_seed = s()
    return w


RESNET18_STAGES = ((64, 1), (128, 2), (256, 2), (512, 2))


def resnet18_shaped_bf16(batch: int = 64, image: int = 224,
                         input_requires_grad: bool = False) -> Workload:
    """Plain ResNet-18-shaped stack of 17 convs each followed by BN-eval, then
    a forward-only global average pool and a trainable 512->1000 Linear.

    Stem 7x7/s2/p3 (3->64); stage 1 four 3x3 convs 64->64, the first with
    stride 2 (standing in for the max-pool); stages 2-4 four 3x3 convs each,
    the first with stride 2.  Convs have no bias.  With the image not
    requiring grad every conv/BN mask is 0 and only the Linear has (W, B).
    `input_requires_grad=True` is the "Input" variant: every conv/BN gets the
    input bit and the Linear gets (I, W, B).
    """
    s = _Seeds(3)
    x_seed = s()
    ib = MASK_INPUT if input_requires_grad else 0
    layers: List[LayerSpec] = []
    shape = (batch, 3, image, image)
    layers.append(_conv("stem", shape, 64, 7, 2, 3, ib, s, bias=False))
    shape = layers[-1].out_shape()
    layers.append(_bn("stem_bn", shape, ib, s))
    cin = 64
    for si, (cout, _) in enumerate(RESNET18_STAGES):
        for j in range(4):
            stride = 2 if j == 0 else 1
            layers.append(_conv(f"s{si + 1}c{j + 1}", shape, cout, 3, stride, 1,
                                ib, s, bias=False))
            shape = layers[-1].out_shape()
            layers.append(_bn(f"s{si + 1}c{j + 1}_bn", shape, ib, s))
            cin = cout
    layers.append(LayerSpec("avgpool", "avgpool", shape, mask=ib))
    feat = layers[-1].out_shape()
    layers.append(_linear("fc", feat[0], feat[1], 1000,
                          ib | MASK_WEIGHT | MASK_BIAS, s,
                          ("kaiming", (feat[1],)), ("kaiming", (feat[1],))))
    name = "resnet18_shaped_bf16" + ("_input" if input_requires_grad else "")
    w = Workload(3, name, "bf16", layers, input_seed=x_seed,
                 note=f"x[{batch},3,{image},{image}], 17 conv+BN-eval, avgpool, fc 512->1000")
    w.grad_seed = s()
    return w


CONV_SWEEP_MASKS = {"00": 0, "10": MASK_INPUT, "01": MASK_WEIGHT | MASK_BIAS,
                    "11": MASK_INPUT | MASK_WEIGHT | MASK_BIAS}


def conv_sweep_bf16(mask_name: str, pointwise: bool = False,
                    batch: int = 32) -> Workload:
    """One bf16 conv on x[32,256,28,28]: 3x3 256->256 pad 1, or the 1x1
    256->1024 pointwise variant; (input, weight) requires-grad combination
    `mask_name` in {"00","10","01","11"}, bias flag = weight flag."""
    s = _Seeds(4)
    x_seed = s()
    mask = CONV_SWEEP_MASKS[mask_name]
    if pointwise:
        layer = _conv("conv1x1", (batch, 256, 28, 28), 1024, 1, 1, 0, mask, s, bias=True)
    else:
        layer = _conv("conv3x3", (batch, 256, 28, 28), 256, 3, 1, 1, mask, s, bias=True)
    w = Workload(4, f"conv_sweep_{'1x1' if pointwise else '3x3'}_{mask_name}_bf16",
                 "bf16", [layer], input_seed=x_seed,
                 note=f"x[{batch},256,28,28], mask (I,W)={mask_name}")
    w.grad_seed = s()
    return w


ENCODER_LINEARS = (("qkv", 768, 2304), ("out", 768, 768),
                   ("ffn_up", 768, 3072), ("ffn_down", 3072, 768))


def encoder_linears_bf16(layers: int = 12, tokens: int = 16 * 512) -> Workload:
    """The Linear layers of a 12-layer hidden-768 encoder on 16x512 tokens,
    weights and biases frozen, grads to the inputs only.  Attention and the
    activation are not on the path: QKV, out and FFN-up each take a fresh
    N(0,1) input; FFN-down takes FFN-up's output."""
    s = _Seeds(5)
    x_seed = s()
    out: List[LayerSpec] = []
    for l in range(layers):
        for nm, kin, nout in ENCODER_LINEARS:
            chained = nm == "ffn_down"
            sp = _linear(f"l{l}.{nm}", tokens, kin, nout, MASK_INPUT, s,
                         ("normal", (0.0, 0.02)), ("normal", (0.0, 0.02)),
                         chained=chained)
            if not chained:
                sp.seeds["x"] = s()
            out.append(sp)
    w = Workload(5, "encoder_linears_bf16", "bf16", out, input_seed=x_seed,
                 note=f"{layers} layers x (768->2304, 768->768, 768->3072, 3072->768), M={tokens}")
    w.grad_seed = s()
    return w


def decoder_convt_bf16(batch: int = 32, mask: int = MASK_INPUT | MASK_WEIGHT | MASK_BIAS) -> Workload:
    """The upsampling path of an image decoder: three bf16 ConvTranspose2d
    layers with bias, 512x14x14 -> 256x28x28 (4x4, stride 2, pad 1) ->
    128x56x56 (4x4, stride 2, pad 1) -> 64x112x112 (2x2, stride 2), every
    layer trained (mask I, W, B by default)."""
    s = _Seeds(6)
    x_seed = s()
    layers = []
    shape = (batch, 512, 14, 14)
    for name, cout, r, pad in (("up1", 256, 4, 1), ("up2", 128, 4, 1), ("up3", 64, 2, 0)):
        layers.append(_convt(name, shape, cout, r, 2, pad, mask, s, bias=True))
        shape = layers[-1].out_shape()
    w = Workload(6, "decoder_convt_bf16", "bf16", layers, input_seed=x_seed,
                 note=f"x[{batch},512,14,14], ConvTranspose2d 4x4/s2/p1 512->256, 4x4/s2/p1 256->128, "
                      f"2x2/s2 128->64")
    w.grad_seed = s()
    return w


def all_workloads() -> Dict[str, Workload]:
    d = {"1": single_conv_f32(), "2": linear_stack_bf16(),
         "3": resnet18_shaped_bf16(), "3b": resnet18_shaped_bf16(input_requires_grad=True),
         "5": encoder_linears_bf16(), "6": decoder_convt_bf16()}
    for mk in CONV_SWEEP_MASKS:
        d[f"4_3x3_{mk}"] = conv_sweep_bf16(mk)
        d[f"4_1x1_{mk}"] = conv_sweep_bf16(mk, pointwise=True)
    return d
