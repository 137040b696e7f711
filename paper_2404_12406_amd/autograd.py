"""PyTorch autograd adapter: the library's layers as torch.autograd.Functions
and nn.Modules, and a converter that swaps them into an existing model
(Sec. 2.2: the method is a drop-in replacement whose forward decides what to
keep from which of its inputs require grad, and whose backward computes only
the gradients autograd asks for).

Each Function derives its mask from ctx.needs_input_grad, runs the forward
through the C ABI and keeps the library's record on ctx -- the record holds
references to exactly the tensors the save rule borrows, so PyTorch's
allocator retains what the ledger reports and nothing else.  Backward hands
grad_y to ms_layer_backward and returns only the requested gradients.

Layout: the 2-D layers take activations in any layout (NCHW, channels-last,
strided views): the library stages what is not channels-last through
transient workspace, and a record borrows the caller's own input.  The
modules keep their weights channels-last (no staging) and return
channels-last outputs, so only the first layer of a stack fed NCHW tensors
pays the staging.  ReLU and dropout work in memory order and take any dense
layout as it is.  The 3-D layers need channels-last-3d tensors and convert an
input that is not (the converted copy is what a record then borrows).  The 1-D layers run as the 2-D ones
with H = 1: their activations [N, C, L] and weights [K, C, R] are kept with
the channel index innermost ([N][L][C], [K][R][C] in memory), so the 4-D
views the library sees are channels-last without a copy.
"""
from __future__ import annotations

from typing import Optional

import torch
from torch import nn

from . import api
from .api import MASK_BIAS, MASK_INPUT, MASK_WEIGHT

__all__ = ["MSConv2d", "MSConvTranspose2d", "MSConv1d", "MSConvTranspose1d", "MSConv3d", "MSConvTranspose3d",
           "MSLinear", "MSBatchNorm2dEval", "MSReLU", "MSDropout", "convert"]


def _cl(t: Optional[torch.Tensor]) -> Optional[torch.Tensor]:
    """Channels-last for 4-D and 5-D tensors (a copy only when needed)."""
    if t is None or t.dim() not in (4, 5):
        return t
    fmt = torch.channels_last if t.dim() == 4 else torch.channels_last_3d
    return t if t.is_contiguous(memory_format=fmt) else t.contiguous(memory_format=fmt)


def _dense(t: torch.Tensor) -> torch.Tensor:
    """t itself when its elements form one dense block (row-major or
    channels-last), else a contiguous copy (for the elementwise layers)."""
    if t.is_contiguous() or (t.dim() == 4 and t.is_contiguous(memory_format=torch.channels_last)):
        return t
    return t.contiguous()


def _as_layout_of(g: torch.Tensor, like) -> torch.Tensor:
    """g with the strides of a tensor of stride `like` (a copy only when they differ)."""
    if g.stride() == tuple(like):
        return g
    out = torch.empty_strided(g.shape, like, dtype=g.dtype, device=g.device)
    out.copy_(g)
    return out


def _versions(rec):
    """(tensor, version counter) of every tensor a record borrows."""
    if rec is None:
        return ()
    out = []
    for v in rec.saved.values():
        for t in (v if isinstance(v, tuple) else (v,)):
            if isinstance(t, torch.Tensor):
                out.append((t, t._version))
    return tuple(out)


def _check_versions(versions):
    for t, v in versions:
        if t._version != v:
            raise RuntimeError("a tensor that the layer's record borrows for backward has been modified by an "
                               f"inplace operation (version {t._version}, expected {v}); the gradient would be "
                               "computed from the modified values")


def _mask(ctx, ix: int, iw: Optional[int] = None, ib: Optional[int] = None) -> int:
    need = ctx.needs_input_grad
    m = MASK_INPUT if need[ix] else 0
    if iw is not None and need[iw]:
        m |= MASK_WEIGHT
    if ib is not None and need[ib]:
        m |= MASK_BIAS
    return m


class _LayerFn(torch.autograd.Function):
    """y = layer(x; W, b) through the C ABI; inputs (spec, x, W, b)."""

    @staticmethod
    def forward(ctx, spec, x, W, b):
        mask = _mask(ctx, 1, 2 if W is not None else None, 3 if b is not None else None)
        y, rec = api.layer_forward(spec, x, W, b, mask)
        ctx.rec = rec
        ctx.has = (W is not None, b is not None)
        # the record borrows these tensors: like autograd's saved tensors,
        # they must not be modified in place before backward
        ctx.versions = _versions(rec)
        return y

    @staticmethod
    def backward(ctx, grad_y):
        rec = ctx.rec
        ctx.rec = None
        if rec is None:
            return None, None, None, None
        _check_versions(ctx.versions)
        gy = grad_y if grad_y.dim() in (2, 4) else _cl(grad_y.contiguous() if grad_y.dim() < 4 else grad_y)
        gx, gw, gb = api.layer_backward(rec, gy)
        rec.free()
        return None, gx, gw, gb


class _ReLUFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        y, rec = api.layer_forward(api.ReLU(), x, mask=_mask(ctx, 0))
        ctx.rec = rec
        ctx.stride = y.stride()
        return y

    @staticmethod
    def backward(ctx, grad_y):
        rec = ctx.rec
        ctx.rec = None
        if rec is None:
            return None
        gx, _, _ = api.layer_backward(rec, _as_layout_of(grad_y, ctx.stride))
        rec.free()
        return gx


class _DropoutFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, p, seed):
        y, rec = api.layer_forward(api.Dropout(p, seed, 0), x, mask=_mask(ctx, 0))
        ctx.rec = rec
        ctx.stride = y.stride()
        return y

    @staticmethod
    def backward(ctx, grad_y):
        rec = ctx.rec
        ctx.rec = None
        if rec is None:
            return None, None, None
        gx, _, _ = api.layer_backward(rec, _as_layout_of(grad_y, ctx.stride))
        rec.free()
        return gx, None, None


class MSConv2d(nn.Module):
    """Conv2d (cross-correlation, zero padding, dilation 1, groups 1) with a
    channels-last weight [K, C, R, S] and optional bias [K]."""

    def __init__(self, weight: torch.Tensor, bias: Optional[torch.Tensor], stride=1, padding=0):
        super().__init__()
        self.weight = weight if isinstance(weight, nn.Parameter) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        with torch.no_grad():
            if not self.weight.is_contiguous(memory_format=torch.channels_last):
                self.weight.data = self.weight.data.contiguous(memory_format=torch.channels_last)
        self.spec = api.Conv2d(stride, padding)

    def forward(self, x):
        return _LayerFn.apply(self.spec, x, self.weight, self.bias)


class MSConvTranspose2d(nn.Module):
    """ConvTranspose2d (dilation 1, groups 1) with a channels-last weight
    [C_in, C_out, R, S], optional bias [C_out] and output padding < stride."""

    def __init__(self, weight: torch.Tensor, bias: Optional[torch.Tensor], stride=1, padding=0,
                 output_padding=0):
        super().__init__()
        self.weight = weight if isinstance(weight, nn.Parameter) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        with torch.no_grad():
            if not self.weight.is_contiguous(memory_format=torch.channels_last):
                self.weight.data = self.weight.data.contiguous(memory_format=torch.channels_last)
        self.spec = api.ConvTranspose2d(stride, padding, output_padding)

    def forward(self, x):
        return _LayerFn.apply(self.spec, x, self.weight, self.bias)


class _Conv3dBase(nn.Module):
    def __init__(self, weight, bias):
        super().__init__()
        self.weight = weight if isinstance(weight, nn.Parameter) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        with torch.no_grad():
            self.weight.data = _cl(self.weight.data)

    def forward(self, x):
        return _LayerFn.apply(self.spec, _cl(x), self.weight, self.bias)


class MSConv3d(_Conv3dBase):
    """Conv3d (zero padding, dilation 1, groups 1), channels-last 3-D
    weight [K, C, T, R, S]."""

    def __init__(self, weight, bias, stride=1, padding=0):
        super().__init__(weight, bias)
        self.spec = api.Conv3d(stride, padding)


class MSConvTranspose3d(_Conv3dBase):
    """ConvTranspose3d (dilation 1, groups 1), channels-last 3-D weight
    [C_in, C_out, T, R, S]."""

    def __init__(self, weight, bias, stride=1, padding=0, output_padding=0):
        super().__init__(weight, bias)
        self.spec = api.ConvTranspose3d(stride, padding, output_padding)


def _channels_inner(t: torch.Tensor) -> torch.Tensor:
    """[A, C, L] with C innermost in memory ([A][L][C])."""
    if t.stride(1) == 1 and t.stride(2) == t.shape[1]:
        return t
    return t.transpose(1, 2).contiguous().transpose(1, 2)


def _first(v):
    return int(v[0]) if isinstance(v, (tuple, list)) else int(v)


class _Conv1dBase(nn.Module):
    def __init__(self, weight, bias):
        super().__init__()
        self.weight = weight if isinstance(weight, nn.Parameter) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        with torch.no_grad():
            self.weight.data = _channels_inner(self.weight.data)

    def forward(self, x):
        y = _LayerFn.apply(self.spec, _cl(_channels_inner(x).unsqueeze(2)), self.weight.unsqueeze(2), self.bias)
        return y.squeeze(2)


class MSConv1d(_Conv1dBase):
    """Conv1d (zero padding, dilation 1, groups 1) as the 2-D convolution
    with H = R = 1: x[N, C, L], weight [K, C, R]."""

    def __init__(self, weight, bias, stride=1, padding=0):
        super().__init__(weight, bias)
        self.spec = api.Conv2d((1, _first(stride)), (0, _first(padding)))


class MSConvTranspose1d(_Conv1dBase):
    """ConvTranspose1d (dilation 1, groups 1) as the 2-D transposed
    convolution with H = R = 1: x[N, C_in, L], weight [C_in, C_out, R]."""

    def __init__(self, weight, bias, stride=1, padding=0, output_padding=0):
        super().__init__(weight, bias)
        self.spec = api.ConvTranspose2d((1, _first(stride)), (0, _first(padding)), (0, _first(output_padding)))


class MSLinear(nn.Module):
    """y = x W^T + b for x[M, K_in] (leading dims are flattened into M)."""

    def __init__(self, weight: torch.Tensor, bias: Optional[torch.Tensor]):
        super().__init__()
        self.weight = weight if isinstance(weight, nn.Parameter) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        self.spec = api.Linear()

    def forward(self, x):
        lead = x.shape[:-1]
        y = _LayerFn.apply(self.spec, x.reshape(-1, x.shape[-1]), self.weight, self.bias)
        return y.reshape(*lead, y.shape[-1])


class MSBatchNorm2dEval(nn.Module):
    """BatchNorm in evaluation mode: fixed running statistics, optional
    affine gamma (weight) and beta (bias)."""

    def __init__(self, weight, bias, running_mean, running_var, eps=1e-5):
        super().__init__()
        self.weight = weight if (weight is None or isinstance(weight, nn.Parameter)) else nn.Parameter(weight)
        self.bias = bias if (bias is None or isinstance(bias, nn.Parameter)) else nn.Parameter(bias)
        self.register_buffer("running_mean", running_mean)
        self.register_buffer("running_var", running_var)
        self.eps = float(eps)

    def forward(self, x):
        spec = api.BatchNormEval(self.running_mean, self.running_var, self.eps)
        return _LayerFn.apply(spec, x, self.weight, self.bias)


class MSReLU(nn.Module):
    """ReLU whose backward keeps one bit per element (Sec. 2.2.2)."""

    def forward(self, x):
        return _ReLUFn.apply(_dense(x))


class MSDropout(nn.Module):
    """Dropout that keeps its generator state, not its mask, and draws the
    mask again in backward (Sec. 2.2.2).  In training mode each call takes a
    fresh 64-bit key from torch's default CPU generator (so torch.manual_seed
    makes runs repeatable; `last_seed` holds the key of the latest call); in
    evaluation mode, or with p = 0, it is the identity.  A dense input (any
    order of its dims) is used as it is, any other one through a contiguous
    copy; the mask is drawn in memory order."""

    def __init__(self, p: float = 0.5):
        super().__init__()
        if not 0.0 <= p <= 1.0:
            raise ValueError("dropout probability must lie in [0, 1]")
        self.p = float(p)
        self.last_seed = None

    def forward(self, x):
        if not self.training or self.p == 0.0:
            return x
        seed = int(torch.randint(0, 2 ** 63 - 1, (), dtype=torch.int64))
        self.last_seed = seed
        return _DropoutFn.apply(_dense(x), self.p, seed)


def _convertible_conv(m) -> bool:
    """groups 1, dilation 1, zero padding given as numbers, fp32 or bf16."""
    return (m.groups == 1 and all(d == 1 for d in m.dilation) and m.padding_mode == "zeros"
            and not isinstance(m.padding, str) and m.weight.dtype in (torch.float32, torch.bfloat16))


def convert(module: nn.Module) -> nn.Module:
    """Replace, in place, every nn.Conv1d/2d/3d and nn.ConvTranspose1d/2d/3d
    (groups 1, dilation 1, zero padding), nn.Linear,
    nn.BatchNorm2d in evaluation mode and nn.ReLU of `module` by the
    library's layers, sharing their parameters and buffers; returns the
    module (Sec. 4: one call swaps every supported layer); nn.Dropout
    becomes MSDropout with the same p and mode.  A BatchNorm2d
    still in training mode is left as it is (its batch statistics make it
    non-linear in x); so is any layer outside those limits."""
    for name, child in list(module.named_children()):
        new = None
        if isinstance(child, nn.Conv2d) and _convertible_conv(child):
            new = MSConv2d(child.weight, child.bias, tuple(child.stride), tuple(child.padding))
        elif isinstance(child, nn.ConvTranspose2d) and _convertible_conv(child):
            new = MSConvTranspose2d(child.weight, child.bias, tuple(child.stride), tuple(child.padding),
                                    tuple(child.output_padding))
        elif isinstance(child, nn.Conv1d) and _convertible_conv(child):
            new = MSConv1d(child.weight, child.bias, child.stride, child.padding)
        elif isinstance(child, nn.ConvTranspose1d) and _convertible_conv(child):
            new = MSConvTranspose1d(child.weight, child.bias, child.stride, child.padding, child.output_padding)
        elif isinstance(child, nn.Conv3d) and _convertible_conv(child):
            new = MSConv3d(child.weight, child.bias, tuple(child.stride), tuple(child.padding))
        elif isinstance(child, nn.ConvTranspose3d) and _convertible_conv(child):
            new = MSConvTranspose3d(child.weight, child.bias, tuple(child.stride), tuple(child.padding),
                                    tuple(child.output_padding))
        elif isinstance(child, nn.Linear):
            new = MSLinear(child.weight, child.bias)
        elif isinstance(child, nn.BatchNorm2d) and not child.training and child.track_running_stats:
            new = MSBatchNorm2dEval(child.weight, child.bias, child.running_mean, child.running_var, child.eps)
        elif isinstance(child, nn.ReLU):
            new = MSReLU()
        elif isinstance(child, nn.Dropout):
            new = MSDropout(child.p)
            new.train(child.training)
        if new is not None:
            setattr(module, name, new)
        else:
            convert(child)
    return module
