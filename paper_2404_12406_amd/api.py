"""Python binding of libmemsave: torch tensors in, the C ABI of
include/memsave.h underneath.  Only argument marshalling happens here; every
arithmetic step runs in the library's HIP kernels.  PyTorch provides device
memory (tensors the caller or this module allocates) and the stream.

    y, rec = layer_forward(Conv2d(stride=1, pad=1), x, W, b, mask=MASK_INPUT)
    gx, gW, gb = layer_backward(rec, grad_y)     # gW, gb are None here

4-D and 2-D tensors may have any strides: channels-last (torch.channels_last)
activations and conv weights and row-major matrices are used in place, any
other layout (NCHW, slices, transposed views) is staged by the library
through transient workspace.  5-D tensors must be channels-last-3d, 1-D
tensors contiguous; ReLU and dropout take any dense layout, with gradients
in the layout of x.  dtypes float32 or bfloat16.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

from . import _lib
from ._lib import (MS_AVGPOOL, MS_BN_EVAL, MS_CONV2D, MS_CONV3D, MS_CONV_TRANSPOSE2D, MS_CONV_TRANSPOSE3D, MS_DROPOUT,
                   MS_LINEAR, MS_RELU, MS_RG_BIAS,
                   MS_RG_INPUT,
                   MS_RG_WEIGHT, MS_SAVED_BITS, MS_SAVED_MEAN, MS_SAVED_VAR, MS_SAVED_W, MS_SAVED_X,
                   MsAccount, MsLayer, MsTensor, check)

MASK_INPUT, MASK_WEIGHT, MASK_BIAS = MS_RG_INPUT, MS_RG_WEIGHT, MS_RG_BIAS
POLICY_SELECTIVE, POLICY_PYTORCH_DEFAULT, POLICY_ALL_TRUE = 0, 1, 2

_DT = {torch.float32: _lib.MS_F32, torch.bfloat16: _lib.MS_BF16}


# ------------------------------------------------------------------ layer specs
@dataclass(frozen=True)
class Conv2d:
    """y = W * x + b (cross-correlation, zero padding, dilation 1, groups 1)."""
    stride: Tuple[int, int] | int = 1
    pad: Tuple[int, int] | int = 0


@dataclass(frozen=True)
class ConvTranspose2d:
    """Transposed convolution (torch.nn.ConvTranspose2d, dilation 1, groups 1)
    with W[C_in, C_out, R, S]: the adjoint of the convolution with that filter,
    stride and pad; out_pad (< stride) extends the output on the high side."""
    stride: Tuple[int, int] | int = 1
    pad: Tuple[int, int] | int = 0
    out_pad: Tuple[int, int] | int = 0


@dataclass(frozen=True)
class Conv3d:
    """3-D Conv2d: x[N,C,D,H,W], W[K,C,T,R,S]; stride and pad are (d, h, w)."""
    stride: Tuple[int, int, int] | int = 1
    pad: Tuple[int, int, int] | int = 0


@dataclass(frozen=True)
class ConvTranspose3d:
    """3-D ConvTranspose2d: x[N,C_in,D,H,W], W[C_in,C_out,T,R,S]; (d, h, w) triples."""
    stride: Tuple[int, int, int] | int = 1
    pad: Tuple[int, int, int] | int = 0
    out_pad: Tuple[int, int, int] | int = 0


@dataclass(frozen=True)
class Linear:
    """y = x W^T + b for x[M, K_in], W[N_out, K_in]."""


@dataclass
class BatchNormEval:
    """y = gamma (x - running_mean) / sqrt(running_var + eps) + beta."""
    running_mean: torch.Tensor
    running_var: torch.Tensor
    eps: float = 1e-5


@dataclass(frozen=True)
class AvgPool:
    """Global average pool x[N, C, H, W] -> y[N, C]."""


@dataclass(frozen=True)
class ReLU:
    """y = max(x, 0); its record keeps one bit per element (y > 0), not y."""


@dataclass(frozen=True)
class Dropout:
    """y = x * m / (1 - p) with the keep mask m drawn from Philox4x32-10
    under key `seed`, starting at block `offset`; its record keeps
    (seed, offset, p), not m, and backward draws m again."""
    p: float = 0.5
    seed: int = 0
    offset: int = 0


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def _triple(v):
    return (int(v),) * 3 if isinstance(v, int) else (int(v[0]), int(v[1]), int(v[2]))


def tensor_desc(t: Optional[torch.Tensor]) -> Optional[MsTensor]:
    """Describe a torch tensor for the C ABI (pointer, dtype, shape, strides)."""
    if t is None:
        return None
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")
    if t.dim() > 5 or t.dim() < 1:
        raise ValueError("tensors must have 1 to 5 dims")
    d = MsTensor()
    d.data = t.data_ptr() if t.numel() > 0 else None
    d.dtype = _DT[t.dtype]
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.stride[i] = t.stride(i)
    return d


def _ptr(d: Optional[MsTensor]):
    return ctypes.byref(d) if d is not None else None


class _LayerDesc:
    """Keeps the MsLayer and the tensors it points to alive together."""

    def __init__(self, spec):
        self.layer = MsLayer()
        self.mean = self.var = None
        self.spec = spec
        if isinstance(spec, Conv2d):
            self.layer.kind = MS_CONV2D
            s, p = _pair(spec.stride), _pair(spec.pad)
            self.layer.stride[0], self.layer.stride[1] = s
            self.layer.pad[0], self.layer.pad[1] = p
        elif isinstance(spec, ConvTranspose2d):
            self.layer.kind = MS_CONV_TRANSPOSE2D
            s, p, o = _pair(spec.stride), _pair(spec.pad), _pair(spec.out_pad)
            self.layer.stride[0], self.layer.stride[1] = s
            self.layer.pad[0], self.layer.pad[1] = p
            self.layer.out_pad[0], self.layer.out_pad[1] = o
        elif isinstance(spec, (Conv3d, ConvTranspose3d)):
            tr = isinstance(spec, ConvTranspose3d)
            self.layer.kind = MS_CONV_TRANSPOSE3D if tr else MS_CONV3D
            s, p = _triple(spec.stride), _triple(spec.pad)
            o = _triple(spec.out_pad) if tr else (0, 0, 0)
            self.layer.stride_d, self.layer.stride[0], self.layer.stride[1] = s
            self.layer.pad_d, self.layer.pad[0], self.layer.pad[1] = p
            self.layer.out_pad_d, self.layer.out_pad[0], self.layer.out_pad[1] = o
        elif isinstance(spec, Linear):
            self.layer.kind = MS_LINEAR
        elif isinstance(spec, BatchNormEval):
            self.layer.kind = MS_BN_EVAL
            self.layer.eps = float(spec.eps)
            self.mean = tensor_desc(spec.running_mean)
            self.var = tensor_desc(spec.running_var)
            self.layer.running_mean = ctypes.pointer(self.mean)
            self.layer.running_var = ctypes.pointer(self.var)
        elif isinstance(spec, AvgPool):
            self.layer.kind = MS_AVGPOOL
        elif isinstance(spec, ReLU):
            self.layer.kind = MS_RELU
        elif isinstance(spec, Dropout):
            self.layer.kind = MS_DROPOUT
        else:
            raise TypeError(f"unknown layer spec {spec!r}")


def _stream(device) -> ctypes.c_void_p:
    if device is None or device.type != "cuda":
        return ctypes.c_void_p(0)
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def output_shape(spec, x: torch.Tensor, W: Optional[torch.Tensor]):
    if isinstance(spec, Conv2d):
        N, _, H, Wd = x.shape
        K, _, R, S = W.shape
        (sh, sw), (ph, pw) = _pair(spec.stride), _pair(spec.pad)
        return (N, K, (H + 2 * ph - R) // sh + 1, (Wd + 2 * pw - S) // sw + 1)
    if isinstance(spec, ConvTranspose2d):
        N, _, H, Wd = x.shape
        _, Co, R, S = W.shape
        (sh, sw), (ph, pw), (oh, ow) = _pair(spec.stride), _pair(spec.pad), _pair(spec.out_pad)
        return (N, Co, (H - 1) * sh - 2 * ph + R + oh, (Wd - 1) * sw - 2 * pw + S + ow)
    if isinstance(spec, Conv3d):
        N, _, D, H, Wd = x.shape
        K, _, T, R, S = W.shape
        s, p = _triple(spec.stride), _triple(spec.pad)
        return (N, K) + tuple((e + 2 * pp - k) // ss + 1 for e, k, ss, pp in zip((D, H, Wd), (T, R, S), s, p))
    if isinstance(spec, ConvTranspose3d):
        N, _, D, H, Wd = x.shape
        _, Co, T, R, S = W.shape
        s, p, o = _triple(spec.stride), _triple(spec.pad), _triple(spec.out_pad)
        return (N, Co) + tuple((e - 1) * ss - 2 * pp + k + oo
                               for e, k, ss, pp, oo in zip((D, H, Wd), (T, R, S), s, p, o))
    if isinstance(spec, Linear):
        return (x.shape[0], W.shape[0])
    if isinstance(spec, BatchNormEval):
        return tuple(x.shape)
    if isinstance(spec, AvgPool):
        return (x.shape[0], x.shape[1])
    if isinstance(spec, (ReLU, Dropout)):
        return tuple(x.shape)
    raise TypeError(spec)


def empty_like_layout(shape, like: torch.Tensor) -> torch.Tensor:
    """Uninitialised tensor of `shape` on like's device in the layout the
    library requires (channels-last for 4-D and 5-D)."""
    if len(shape) == 4:
        return torch.empty(shape, dtype=like.dtype, device=like.device, memory_format=torch.channels_last)
    if len(shape) == 5:
        return torch.empty(shape, dtype=like.dtype, device=like.device, memory_format=torch.channels_last_3d)
    return torch.empty(shape, dtype=like.dtype, device=like.device)


# ------------------------------------------------------------------ records
class Record:
    """A saved-tensor record: the C record plus torch references to exactly
    the tensors it borrows (so the caching allocator sees the same retained
    bytes as the ledger)."""

    def __init__(self, handle: ctypes.c_void_p, desc: _LayerDesc, x, W, b, y_shape, y_like, bits=None):
        self._h = handle
        self._desc = desc
        acct = self.account()
        self.mask = acct["mask"]
        bor = acct["borrowed"]
        self._keep = {}
        if bor & MS_SAVED_BITS:
            self._keep["bits"] = bits
        if bor & MS_SAVED_X:
            self._keep["x"] = x
        if bor & MS_SAVED_W:
            self._keep["W"] = W
        if bor & (MS_SAVED_MEAN | MS_SAVED_VAR):
            self._keep["stats"] = (desc.spec.running_mean, desc.spec.running_var)
        self._x_meta = (tuple(x.shape), x.dtype, x.device, tuple(x.stride()))
        self._elementwise = isinstance(desc.spec, (ReLU, Dropout))
        self._w_meta = (tuple(W.shape), W.dtype) if W is not None else None
        self._b_meta = (tuple(b.shape), b.dtype) if b is not None else None
        self.y_shape = y_shape
        self.consumed = False

    @property
    def saved(self):
        return dict(self._keep)

    def account(self) -> dict:
        a = MsAccount()
        check(_lib.load().ms_record_account(self._h, ctypes.byref(a)), "ms_record_account")
        return a.as_dict()

    def release_refs(self):
        self._keep = {}

    def free(self):
        if self._h is not None:
            lib = _lib._lib
            if lib is not None:
                lib.ms_record_free(self._h)
            self._h = None
            self._keep = {}

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def _on_gpu(*ts):
    """The library dereferences device pointers only: refuse host tensors."""
    dev = None
    for t in ts:
        if t is None:
            continue
        if t.device.type != "cuda":
            raise TypeError("libmemsave computes on the GPU only; got a tensor on " + str(t.device))
        if dev is not None and t.device != dev:
            raise ValueError("all tensors of one call must be on the same device")
        dev = t.device
    if dev is not None:
        torch.cuda.set_device(dev)


def relu_mask_bytes(numel: int) -> int:
    """Bytes of the 1-bit mask a ReLU record keeps for `numel` elements."""
    return int(_lib.load().ms_relu_mask_bytes(int(numel)))


def relu_mask_buffer(x: torch.Tensor) -> torch.Tensor:
    """A device buffer for the 1-bit mask of a ReLU over x (int32 words)."""
    return torch.empty(relu_mask_bytes(x.numel()) // 4, dtype=torch.int32, device=x.device)


def _relu_forward(lib, x, y, bits, mask):
    h = ctypes.c_void_p()
    st = lib.ms_relu_forward(_ptr(tensor_desc(x)), _ptr(tensor_desc(y)),
                             ctypes.c_void_p(bits.data_ptr() if bits is not None and bits.numel() else None),
                             int(mask), ctypes.byref(h), _stream(x.device))
    check(st, "ms_relu_forward")
    return h


def dropout_blocks(numel: int) -> int:
    """Generator blocks one dropout call over `numel` elements consumes."""
    return int(_lib.load().ms_dropout_blocks(int(numel)))


def _dropout_forward(lib, spec, x, y, mask):
    h = ctypes.c_void_p()
    st = lib.ms_dropout_forward(_ptr(tensor_desc(x)), _ptr(tensor_desc(y)), float(spec.p), int(spec.seed),
                                int(spec.offset), int(mask), ctypes.byref(h), _stream(x.device))
    check(st, "ms_dropout_forward")
    return h


def layer_forward(spec, x: torch.Tensor, W: Optional[torch.Tensor] = None, b: Optional[torch.Tensor] = None,
                  mask: int = 0, y: Optional[torch.Tensor] = None):
    """Run the layer's forward kernel on the current stream; return (y, record).
    record is None when mask == 0 (nothing is saved).  A ReLU with the INPUT
    bit gets a fresh 1-bit mask buffer, owned by its record."""
    lib = _lib.load()
    if isinstance(spec, ReLU):
        if W is not None or b is not None:
            raise TypeError("ReLU takes no W or b")
        _on_gpu(x, y)
        if y is None:
            y = torch.empty_like(x)   # x's (dense) layout: the mask runs in memory order
        bits = relu_mask_buffer(x) if mask & MASK_INPUT else None
        h = _relu_forward(lib, x, y, bits, mask)
        if not h.value:
            return y, None
        return y, Record(h, _LayerDesc(spec), x, None, None, tuple(y.shape), y, bits)
    if isinstance(spec, Dropout):
        if W is not None or b is not None:
            raise TypeError("dropout takes no W or b")
        _on_gpu(x, y)
        if y is None:
            y = torch.empty_like(x)   # x's (dense) layout: the mask runs in memory order
        h = _dropout_forward(lib, spec, x, y, mask)
        if not h.value:
            return y, None
        return y, Record(h, _LayerDesc(spec), x, None, None, tuple(y.shape), y)
    desc = _LayerDesc(spec)
    extra = (spec.running_mean, spec.running_var) if isinstance(spec, BatchNormEval) else ()
    _on_gpu(x, W, b, y, *extra)
    if y is None:
        y = empty_like_layout(output_shape(spec, x, W), x)
    dx, dw, db, dy = tensor_desc(x), tensor_desc(W), tensor_desc(b), tensor_desc(y)
    h = ctypes.c_void_p()
    st = lib.ms_layer_forward(ctypes.byref(desc.layer), _ptr(dx), _ptr(dw), _ptr(db), int(mask), _ptr(dy),
                              ctypes.byref(h), _stream(x.device))
    check(st, "ms_layer_forward")
    if not h.value:
        return y, None
    return y, Record(h, desc, x, W, b, tuple(y.shape), y)


def layer_backward(rec: Record, grad_y: torch.Tensor, grad_x: Optional[torch.Tensor] = None,
                   grad_W: Optional[torch.Tensor] = None, grad_b: Optional[torch.Tensor] = None):
    """Write exactly the requested gradients; return (grad_x, grad_W, grad_b)
    with None for every gradient the record's mask does not request.
    Gradient buffers not passed in are allocated here."""
    lib = _lib.load()
    _on_gpu(grad_y, grad_x, grad_W, grad_b)
    m = rec.mask
    if m & MASK_INPUT and grad_x is None:
        if rec._elementwise:   # memory order: the gradient in x's layout
            grad_x = torch.empty_strided(rec._x_meta[0], rec._x_meta[3], dtype=grad_y.dtype, device=grad_y.device)
        else:
            grad_x = empty_like_layout(rec._x_meta[0], grad_y)
    if m & MASK_WEIGHT and grad_W is None:
        grad_W = empty_like_layout(rec._w_meta[0], grad_y)
    if m & MASK_BIAS and grad_b is None:
        grad_b = torch.empty(rec._b_meta[0], dtype=grad_y.dtype, device=grad_y.device)
    gy, gx, gw, gb = tensor_desc(grad_y), tensor_desc(grad_x), tensor_desc(grad_W), tensor_desc(grad_b)
    st = lib.ms_layer_backward(rec._h, _ptr(gy), _ptr(gx), _ptr(gw), _ptr(gb), _stream(grad_y.device))
    check(st, "ms_layer_backward")
    rec.consumed = True
    rec.release_refs()
    return grad_x, grad_W, grad_b


def policy_account(spec, x: torch.Tensor, W: Optional[torch.Tensor] = None, b: Optional[torch.Tensor] = None,
                   mask: int = 0, policy: int = POLICY_SELECTIVE) -> dict:
    """Accounting a forward call would produce under `policy`; launches nothing."""
    lib = _lib.load()
    desc = _LayerDesc(spec)
    a = MsAccount()
    st = lib.ms_policy_account(ctypes.byref(desc.layer), _ptr(tensor_desc(x)), _ptr(tensor_desc(W)),
                               _ptr(tensor_desc(b)), int(mask), int(policy), ctypes.byref(a))
    check(st, "ms_policy_account")
    return a.as_dict()


def ledger_read() -> Tuple[int, int]:
    live, peak = ctypes.c_uint64(), ctypes.c_uint64()
    check(_lib.load().ms_ledger_read(ctypes.byref(live), ctypes.byref(peak)), "ms_ledger_read")
    return int(live.value), int(peak.value)


def ledger_reset():
    check(_lib.load().ms_ledger_reset(), "ms_ledger_reset")


PROF_FWD, PROF_DGRAD, PROF_WGRAD, PROF_BN, PROF_ACT, PROF_RED = 1, 2, 4, 8, 16, 32
PROF_ALL = 63


def profile_start(kinds: int):
    """Arm HIP-event timing of the selected kernel kinds (PROF_* bits)."""
    check(_lib.load().ms_profile_start(int(kinds)), "ms_profile_start")


def profile_read(kind: int):
    """(launches, total milliseconds) of one kernel kind since profile_start."""
    n, t = ctypes.c_uint64(), ctypes.c_double()
    check(_lib.load().ms_profile_read(int(kind), ctypes.byref(n), ctypes.byref(t)), "ms_profile_read")
    return int(n.value), float(t.value)


def version() -> str:
    return _lib.load().ms_version().decode()


# ------------------------------------------------------------------ prepared calls
class PreparedLayer:
    """One layer call with its C descriptors built once, for tight loops.

    forward() enqueues ms_layer_forward on the current stream and keeps the
    raw record; backward() enqueues ms_layer_backward for it and frees it.
    A Dropout spec's seed and offset are part of the prepared call, so every
    forward draws the same mask (prepare a new call, or use layer_forward,
    to draw another).
    The object holds references to every tensor it describes, so nothing it
    points to can be freed while it exists."""

    def __init__(self, spec, x, W=None, b=None, mask: int = 0, y=None,
                 grad_y=None, grad_x=None, grad_W=None, grad_b=None):
        extra = (spec.running_mean, spec.running_var) if isinstance(spec, BatchNormEval) else ()
        _on_gpu(x, W, b, y, grad_y, grad_x, grad_W, grad_b, *extra)
        self.lib = _lib.load()
        self.desc = _LayerDesc(spec)
        if y is None:
            y = torch.empty_like(x) if isinstance(spec, (ReLU, Dropout)) else empty_like_layout(output_shape(spec, x, W), x)
        self.tensors = (x, W, b, y, grad_y, grad_x, grad_W, grad_b)
        self.y = y
        self.mask = int(mask)
        self.relu = isinstance(spec, ReLU)
        self.dropout = spec if isinstance(spec, Dropout) else None
        # a ReLU's 1-bit mask lives as long as this object (reused by every forward)
        self.bits = relu_mask_buffer(x) if self.relu and self.mask & MASK_INPUT else None
        self._d = [tensor_desc(t) for t in self.tensors]
        self._fa = (ctypes.byref(self.desc.layer),) + tuple(_ptr(d) for d in self._d[:3])
        self._fy = _ptr(self._d[3])
        self._ba = tuple(_ptr(d) for d in self._d[4:])
        self._h = ctypes.c_void_p()
        self._hp = ctypes.byref(self._h)
        self._stream = _stream(x.device)
        self._free = self.lib.ms_record_free

    def forward(self):
        if self._h.value:
            self._free(self._h)
            self._h.value = None
        if self.relu:
            bits = ctypes.c_void_p(self.bits.data_ptr() if self.bits is not None and self.bits.numel() else None)
            check(self.lib.ms_relu_forward(self._fa[1], self._fy, bits, self.mask, self._hp, self._stream),
                  "ms_relu_forward")
            return
        if self.dropout is not None:
            d = self.dropout
            check(self.lib.ms_dropout_forward(self._fa[1], self._fy, float(d.p), int(d.seed), int(d.offset),
                                              self.mask, self._hp, self._stream), "ms_dropout_forward")
            return
        check(self.lib.ms_layer_forward(*self._fa, self.mask, self._fy, self._hp, self._stream),
              "ms_layer_forward")

    def backward(self):
        if not self._h.value:
            raise RuntimeError("backward without a live record")
        check(self.lib.ms_layer_backward(self._h, *self._ba, self._stream), "ms_layer_backward")
        self._free(self._h)
        self._h.value = None

    def account(self) -> dict:
        a = MsAccount()
        check(self.lib.ms_record_account(self._h, ctypes.byref(a)), "ms_record_account")
        return a.as_dict()

    def __del__(self):
        try:
            if self._h.value:
                self._free(self._h)
        except Exception:
            pass
