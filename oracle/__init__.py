"""CPU oracle of the selective-differentiation layers (TEST INFRASTRUCTURE).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package.  It is the plain definition of what the GPU library
computes (Sec. 2.2.1 and App. C of the paper), evaluated in float64 by the C
loops of oracle.c, plus the closed-form save rule in `oracle.policy`.  It
shares no code with the HIP library and never reads anything the GPU wrote.

All arrays are numpy arrays in the logical PyTorch order (conv/BN/avgpool:
N,C,H,W; conv weight: K,C,R,S; linear: X[M,K_in], W[N_out,K_in]); inputs of
any float dtype are widened to float64, outputs are float64.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

from . import build as _build

__all__ = [
    "conv2d_forward", "conv2d_forward_at", "conv2d_input_grad", "conv2d_input_grad_at",
    "conv2d_weight_grad", "conv2d_weight_grad_at", "conv2d_bias_grad", "conv_out_hw",
    "convt2d_out_hw", "convt2d_forward", "convt2d_forward_at", "convt2d_input_grad", "convt2d_input_grad_at",
    "convt2d_weight_grad", "convt2d_weight_grad_at", "convt2d_bias_grad",
    "linear_forward", "linear_forward_at", "linear_input_grad", "linear_input_grad_at",
    "linear_weight_grad", "linear_weight_grad_at", "linear_bias_grad",
    "bn_eval_forward", "bn_eval_backward", "avgpool_forward", "avgpool_backward",
    "relu_forward", "relu_mask_bits", "relu_backward", "relu_mask_nbytes", "memory_order",
    "philox4x32_10", "dropout_threshold", "dropout_scale", "dropout_words", "dropout_keep", "dropout_forward",
    "dropout_backward", "conv3d_out", "conv3d_forward", "conv3d_input_grad", "conv3d_weight_grad", "bias_grad5",
    "convt3d_out", "convt3d_forward", "convt3d_input_grad", "convt3d_weight_grad",
    "round_to", "rel_err",
]

_lib = None
_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.c_int64


def _load():
    global _lib
    if _lib is None:
        path = _build.build(force=False)
        _lib = ctypes.CDLL(path)
    return _lib


def _d(a):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    if a is None:
        return ctypes.cast(None, _D)
    return a.ctypes.data_as(_D)


def _idx(idx, width):
    a = np.ascontiguousarray(idx, dtype=np.int64).reshape(-1, width)
    return a, a.shape[0]


def conv_out_hw(H, W, R, S, stride, pad):
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    if P < 1 or Q < 1:
        raise ValueError("convolution output would be empty")
    return P, Q


def _conv_args(x_shape, w_shape, stride, pad):
    N, C, H, W = x_shape
    K, C2, R, S = w_shape
    if C2 != C:
        raise ValueError("channel mismatch")
    return [_I(v) for v in (N, C, H, W, K, R, S, stride[0], stride[1], pad[0], pad[1])]


# ----------------------------------------------------------------- conv_transpose2d
def convt2d_out_hw(H, W, R, S, stride, pad, out_pad=(0, 0)):
    """Output extent of the transposed convolution (torch.nn.ConvTranspose2d,
    dilation 1): (H-1) stride - 2 pad + R + out_pad."""
    if not (0 <= out_pad[0] < stride[0] and 0 <= out_pad[1] < stride[1]):
        raise ValueError("output padding must satisfy 0 <= out_pad < stride")
    Ho = (H - 1) * stride[0] - 2 * pad[0] + R + out_pad[0]
    Wo = (W - 1) * stride[1] - 2 * pad[1] + S + out_pad[1]
    if Ho < 1 or Wo < 1:
        raise ValueError("transposed convolution output would be empty")
    return Ho, Wo


def _convt_args(x_shape, w_shape, stride, pad, out_pad):
    N, Ci, H, W = x_shape
    Ci2, Co, R, S = w_shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Ho, Wo = convt2d_out_hw(H, W, R, S, stride, pad, out_pad)
    return [_I(v) for v in (N, Ci, H, W, Co, R, S, stride[0], stride[1], pad[0], pad[1])], (Ho, Wo)


def convt2d_forward(x, w, b=None, stride=(1, 1), pad=(0, 0), out_pad=(0, 0)):
    """Transposed convolution, x[N,Ci,H,W], W[Ci,Co,R,S]: every input pixel
    scatters x W through each tap to the output pixel h*stride - pad + r
    (Sec. 2.2.1 names the layer; App. B lists it)."""
    x, w, b = _d(x), _d(w), _d(b)
    args, (Ho, Wo) = _convt_args(x.shape, w.shape, stride, pad, out_pad)
    y = np.empty((x.shape[0], w.shape[1], Ho, Wo), np.float64)
    _load().orc_convt2d_forward(_p(x), _p(w), _p(b), _p(y), *args, _I(Ho), _I(Wo))
    return y


def convt2d_forward_at(x, w, b, stride, pad, out_pad, idx):
    """Forward values at sampled (n, o, h', w') coordinates, gathered."""
    x, w, b = _d(x), _d(w), _d(b)
    args, _ = _convt_args(x.shape, w.shape, stride, pad, out_pad)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_convt2d_forward_at(_p(x), _p(w), _p(b), *args,
                                   ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def convt2d_input_grad(dy, w, x_shape, stride=(1, 1), pad=(0, 0), out_pad=(0, 0)):
    """dx[n,i,h,w] = sum_{o,r,s} W[i,o,r,s] dy[n,o,h*sh-ph+r,w*sw-pw+s] (needs W only)."""
    dy, w = _d(dy), _d(w)
    args, (Ho, Wo) = _convt_args(x_shape, w.shape, stride, pad, out_pad)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().orc_convt2d_input_grad(_p(dy), _p(w), _p(dx), *args, _I(Ho), _I(Wo))
    return dx


def convt2d_input_grad_at(dy, w, x_shape, stride, pad, out_pad, idx):
    dy, w = _d(dy), _d(w)
    args, (Ho, Wo) = _convt_args(x_shape, w.shape, stride, pad, out_pad)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_convt2d_input_grad_at(_p(dy), _p(w), *args, _I(Ho), _I(Wo),
                                      ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def convt2d_weight_grad(dy, x, w_shape, stride=(1, 1), pad=(0, 0), out_pad=(0, 0)):
    """dW[i,o,r,s] = sum_{n,h,w} x[n,i,h,w] dy[n,o,h*sh-ph+r,w*sw-pw+s] (needs x only)."""
    dy, x = _d(dy), _d(x)
    args, (Ho, Wo) = _convt_args(x.shape, w_shape, stride, pad, out_pad)
    dw = np.empty(tuple(w_shape), np.float64)
    _load().orc_convt2d_weight_grad(_p(dy), _p(x), _p(dw), *args, _I(Ho), _I(Wo))
    return dw


def convt2d_weight_grad_at(dy, x, w_shape, stride, pad, out_pad, idx):
    dy, x = _d(dy), _d(x)
    args, (Ho, Wo) = _convt_args(x.shape, w_shape, stride, pad, out_pad)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_convt2d_weight_grad_at(_p(dy), _p(x), *args, _I(Ho), _I(Wo),
                                       ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def convt2d_bias_grad(dy):
    """db[o] = sum over (n, h', w') of dy: the same column sum as any bias."""
    return conv2d_bias_grad(dy)


# ----------------------------------------------------------------- conv2d
def conv2d_forward(x, w, b=None, stride=(1, 1), pad=(0, 0)):
    """y = W * x + b (cross-correlation, zero padding), Sec. 2.2.1."""
    x, w, b = _d(x), _d(w), _d(b)
    N, _, H, W = x.shape
    K, _, R, S = w.shape
    P, Q = conv_out_hw(H, W, R, S, stride, pad)
    y = np.empty((N, K, P, Q), np.float64)
    _load().orc_conv2d_forward(_p(x), _p(w), _p(b), _p(y), *_conv_args(x.shape, w.shape, stride, pad))
    return y


def conv2d_forward_at(x, w, b, stride, pad, idx):
    """Forward values at sampled (n, k, p, q) coordinates."""
    x, w, b = _d(x), _d(w), _d(b)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_conv2d_forward_at(_p(x), _p(w), _p(b), *_conv_args(x.shape, w.shape, stride, pad),
                                  ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def conv2d_input_grad(dy, w, x_shape, stride=(1, 1), pad=(0, 0)):
    """dx for grad dy (needs W only), as the adjoint scatter of the forward."""
    dy, w = _d(dy), _d(w)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().orc_conv2d_input_grad(_p(dy), _p(w), _p(dx), *_conv_args(x_shape, w.shape, stride, pad))
    return dx


def conv2d_input_grad_at(dy, w, x_shape, stride, pad, idx):
    """dx at sampled (n, c, h, w) coordinates, gathered entry by entry."""
    dy, w = _d(dy), _d(w)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_conv2d_input_grad_at(_p(dy), _p(w), *_conv_args(x_shape, w.shape, stride, pad),
                                     ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def conv2d_weight_grad(dy, x, w_shape, stride=(1, 1), pad=(0, 0)):
    """dW for grad dy (needs x only)."""
    dy, x = _d(dy), _d(x)
    dw = np.empty(tuple(w_shape), np.float64)
    _load().orc_conv2d_weight_grad(_p(dy), _p(x), _p(dw), *_conv_args(x.shape, w_shape, stride, pad))
    return dw


def conv2d_weight_grad_at(dy, x, w_shape, stride, pad, idx):
    """dW at sampled (k, c, r, s) coordinates."""
    dy, x = _d(dy), _d(x)
    ia, n = _idx(idx, 4)
    out = np.empty(n, np.float64)
    _load().orc_conv2d_weight_grad_at(_p(dy), _p(x), *_conv_args(x.shape, w_shape, stride, pad),
                                      ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def conv2d_bias_grad(dy):
    dy = _d(dy)
    N, K, P, Q = dy.shape
    db = np.empty(K, np.float64)
    _load().orc_conv2d_bias_grad(_p(dy), _p(db), _I(N), _I(K), _I(P), _I(Q))
    return db


# ----------------------------------------------------------------- linear
def linear_forward(X, W, b=None):
    """Y = X W^T + b: the layer y = W x + b applied to every row of X."""
    X, W, b = _d(X), _d(W), _d(b)
    M, Kin = X.shape
    Nout, K2 = W.shape
    if K2 != Kin:
        raise ValueError("feature mismatch")
    Y = np.empty((M, Nout), np.float64)
    _load().orc_linear_forward(_p(X), _p(W), _p(b), _p(Y), _I(M), _I(Kin), _I(Nout))
    return Y


def linear_forward_at(X, W, b, idx):
    X, W, b = _d(X), _d(W), _d(b)
    ia, n = _idx(idx, 2)
    out = np.empty(n, np.float64)
    _load().orc_linear_forward_at(_p(X), _p(W), _p(b), _I(X.shape[0]), _I(X.shape[1]), _I(W.shape[0]),
                                  ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def linear_input_grad(dY, W):
    dY, W = _d(dY), _d(W)
    M, Nout = dY.shape
    Kin = W.shape[1]
    dX = np.empty((M, Kin), np.float64)
    _load().orc_linear_input_grad(_p(dY), _p(W), _p(dX), _I(M), _I(Kin), _I(Nout))
    return dX


def linear_input_grad_at(dY, W, idx):
    dY, W = _d(dY), _d(W)
    ia, n = _idx(idx, 2)
    out = np.empty(n, np.float64)
    _load().orc_linear_input_grad_at(_p(dY), _p(W), _I(dY.shape[0]), _I(W.shape[1]), _I(W.shape[0]),
                                     ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def linear_weight_grad(dY, X):
    dY, X = _d(dY), _d(X)
    M, Nout = dY.shape
    Kin = X.shape[1]
    dW = np.empty((Nout, Kin), np.float64)
    _load().orc_linear_weight_grad(_p(dY), _p(X), _p(dW), _I(M), _I(Kin), _I(Nout))
    return dW


def linear_weight_grad_at(dY, X, idx):
    dY, X = _d(dY), _d(X)
    ia, n = _idx(idx, 2)
    out = np.empty(n, np.float64)
    _load().orc_linear_weight_grad_at(_p(dY), _p(X), _I(dY.shape[0]), _I(X.shape[1]), _I(dY.shape[1]),
                                      ia.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _I(n), _p(out))
    return out


def linear_bias_grad(dY):
    dY = _d(dY)
    M, Nout = dY.shape
    db = np.empty(Nout, np.float64)
    _load().orc_linear_bias_grad(_p(dY), _p(db), _I(M), _I(Nout))
    return db


# ----------------------------------------------------------------- BN eval
def _ncl(shape):
    if len(shape) == 2:
        return shape[0], shape[1], 1
    N, C = shape[0], shape[1]
    L = 1
    for s in shape[2:]:
        L *= s
    return N, C, L


def bn_eval_forward(x, mean, var, gamma=None, beta=None, eps=1e-5):
    """y = gamma (x - mu_hat) / sqrt(sigma_hat^2 + eps) + beta per channel (App. C)."""
    x, mean, var, gamma, beta = map(_d, (x, mean, var, gamma, beta))
    y = np.empty(x.shape, np.float64)
    N, C, L = _ncl(x.shape)
    _load().orc_bn_eval_forward(_p(x), _p(mean), _p(var), _p(gamma), _p(beta),
                                ctypes.c_double(eps), _p(y), _I(N), _I(C), _I(L))
    return y


def bn_eval_backward(dy, x, mean, var, gamma=None, eps=1e-5,
                     want_dx=True, want_dgamma=True, want_dbeta=True):
    """(dx, dgamma, dbeta) of BN-eval; each None unless requested.  x may be
    None when dgamma is not requested (the input gradient does not need it)."""
    dy, x, mean, var, gamma = map(_d, (dy, x, mean, var, gamma))
    N, C, L = _ncl(dy.shape)
    if want_dgamma and x is None:
        raise ValueError("dgamma needs x")
    dx = np.empty(dy.shape, np.float64) if want_dx else None
    dg = np.empty(C, np.float64) if want_dgamma else None
    dbt = np.empty(C, np.float64) if want_dbeta else None
    xx = x if x is not None else dy  # never read when dgamma is not requested
    _load().orc_bn_eval_backward(_p(dy), _p(xx), _p(mean), _p(var), _p(gamma), ctypes.c_double(eps),
                                 _p(dx), _p(dg), _p(dbt), _I(N), _I(C), _I(L))
    return dx, dg, dbt


# ----------------------------------------------------------------- avgpool
def avgpool_forward(x):
    x = _d(x)
    N, C, L = _ncl(x.shape)
    y = np.empty((N, C), np.float64)
    _load().orc_avgpool_forward(_p(x), _p(y), _I(N), _I(C), _I(L))
    return y


def avgpool_backward(dy, x_shape):
    dy = _d(dy)
    N, C, L = _ncl(x_shape)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().orc_avgpool_backward(_p(dy), _p(dx), _I(N), _I(C), _I(L))
    return dx


# ----------------------------------------------------------------- rounding, error
# ---------------------------------------------------------------- ReLU (Sec. 2.2.2)
# The activation whose stored output would keep the next linear layer's input
# alive; its input gradient needs only which outputs are positive, so the
# paper's version keeps a boolean mask of the output instead (one bit per
# element here).  Written element by element from the definition:
#   y = x if x >= 0 else 0      (a NaN stays NaN, as torch.relu keeps it)
#   bit i = not (y_i <= 0)      in memory order, 8 per byte, bit e of byte j
#                                is element 8 j + e; 4 * ceil(n / 32) bytes
#   dx_i = dy_i if bit i else 0
# (The paper does not treat NaN; a NaN output passes its gradient, as
# PyTorch's ReLU backward does, whose layer this one replaces.)
def relu_forward(x):
    """y = max(x, 0) elementwise, exact (no rounding: y is a copy of x or 0)."""
    x = np.asarray(x, dtype=np.float64)
    y = x.copy()
    y[x < 0] = 0.0
    return y


def memory_order(a, layout: str = "plain"):
    """The elements of a logical-order array in the library's memory order:
    "nhwc" for 4-D channels-last activations, "plain" for row-major."""
    a = np.asarray(a)
    if layout == "nhwc":
        return np.transpose(a, (0, 2, 3, 1)).reshape(-1)
    return a.reshape(-1)


def relu_mask_nbytes(n: int) -> int:
    return 4 * ((int(n) + 31) // 32) if n > 0 else 0


def relu_mask_bits(x_mem):
    """The 1-bit mask of a ReLU over the 1-D memory-order elements x_mem,
    as uint8 bytes (bit e of byte j = not (relu(x)[8 j + e] <= 0))."""
    x_mem = np.asarray(x_mem, dtype=np.float64).reshape(-1)
    n = x_mem.size
    out = np.zeros(relu_mask_nbytes(n), dtype=np.uint8)
    pos = ~(relu_forward(x_mem) <= 0)
    for i in np.nonzero(pos)[0]:
        out[i // 8] |= np.uint8(1 << (int(i) % 8))
    return out


def relu_backward(dy, x):
    """dx = dy where not relu(x) <= 0, else 0 (same logical shape as x)."""
    dy = np.asarray(dy, dtype=np.float64)
    pos = ~(relu_forward(x) <= 0)
    return np.where(pos, dy, 0.0)


def round_to(a, dtype):
    """Round float64 values once to 'f32' or 'bf16' (ties to even); float64 out."""
    a = np.array(a, dtype=np.float64, copy=True, order="C")
    code = {"f32": 0, "bf16": 1}[dtype]
    _load().orc_round(_p(a), _I(a.size), ctypes.c_int(code))
    return a


def rel_err(got, ref):
    """Normwise max relative error max|got - ref| / max|ref|; inf on any
    non-finite value in `got`."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.shape != ref.shape:
        raise ValueError(f"shape mismatch {got.shape} vs {ref.shape}")
    if got.size == 0:
        return 0.0
    if not np.all(np.isfinite(got)):
        return float("inf")
    den = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(got - ref)))
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den


def threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().orc_threads())


# ----------------------------------------------------------------- dropout
_U32 = ctypes.POINTER(ctypes.c_uint32)


def philox4x32_10(ctr, key):
    """One Philox4x32-10 block (Salmon et al., SC 2011): 4 counter words and
    2 key words in, 4 words out."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    assert c.shape == (4,) and k.shape == (2,)
    out = np.empty(4, np.uint32)
    _load().orc_philox4x32_10(c.ctypes.data_as(_U32), k.ctypes.data_as(_U32), out.ctypes.data_as(_U32))
    return out


def dropout_threshold(p):
    """(thresh, drop_all) of drop probability p taken as a float32: an element
    is kept iff its stream word is >= floor(p * 2^32); p = 1 drops every
    element (Sec. 2.2.2 leaves the generator and the draw to the
    implementation)."""
    p32 = float(np.float32(p))
    if not (0.0 <= p32 <= 1.0):
        raise ValueError("p must lie in [0, 1]")
    if p32 == 1.0:
        return 0, True
    return int(math.floor(p32 * 4294967296.0)), False


def dropout_scale(p):
    """1 / (1 - p) for p taken as a float32, rounded to float32 (0 when p = 1)."""
    p32 = float(np.float32(p))
    return 0.0 if p32 == 1.0 else float(np.float32(1.0 / (1.0 - p32)))


def dropout_words(n, seed, offset=0):
    """The n stream words of one call (element i: word i mod 4 of block
    offset + i // 4 under key `seed`)."""
    u = np.empty(int(n), np.uint32)
    if n > 0:
        _load().orc_dropout_words(_I(int(n)), ctypes.c_uint64(int(seed)), ctypes.c_uint64(int(offset)),
                                  u.ctypes.data_as(_U32))
    return u


def dropout_keep(n, p, seed, offset=0):
    """Which of n elements (memory order) are kept."""
    t, drop_all = dropout_threshold(p)
    if drop_all:
        return np.zeros(int(n), bool)
    return dropout_words(n, seed, offset) >= np.uint32(t)


def dropout_forward(x_mem, p, seed, offset=0):
    """y = x * m / (1 - p) over a flat array in memory order, m the kept
    mask: each element is multiplied by 1/(1-p) (float32) when kept and by 0
    when dropped; p = 1 gives zeros."""
    x = np.asarray(x_mem, dtype=np.float64).reshape(-1)
    t, drop_all = dropout_threshold(p)
    if drop_all:
        return np.zeros_like(x)
    s = np.where(dropout_keep(x.size, p, seed, offset), dropout_scale(p), 0.0)
    return x * s


def dropout_backward(dy_mem, p, seed, offset=0):
    """dx = dy * m / (1 - p) with the mask drawn again from the same counters
    (the forward map is linear with that diagonal Jacobian)."""
    return dropout_forward(dy_mem, p, seed, offset)


# ----------------------------------------------------------------- 3-D convolution and its transpose
def _g3(N, C, D, H, W, K, T, R, S, Do, P, Q, stride, pad):
    return np.array([N, C, D, H, W, K, T, R, S, Do, P, Q, stride[0], stride[1], stride[2],
                     pad[0], pad[1], pad[2]], np.int64)


def _gp(g):
    return g.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def conv3d_out(D, H, W, T, R, S, stride, pad):
    out = tuple((e + 2 * p - k) // s + 1 for e, k, s, p in zip((D, H, W), (T, R, S), stride, pad))
    if min(out) < 1:
        raise ValueError("convolution output would be empty")
    return out


def conv3d_forward(x, w, b=None, stride=(1, 1, 1), pad=(0, 0, 0)):
    """3-D cross-correlation with zero padding (torch.nn.Conv3d, App. B):
    x[N,C,D,H,W], W[K,C,T,R,S]."""
    x, w, b = _d(x), _d(w), _d(b)
    N, C, D, H, W = x.shape
    K, C2, T, R, S = w.shape
    if C2 != C:
        raise ValueError("channel mismatch")
    Do, P, Q = conv3d_out(D, H, W, T, R, S, stride, pad)
    g = _g3(N, C, D, H, W, K, T, R, S, Do, P, Q, stride, pad)
    y = np.empty((N, K, Do, P, Q), np.float64)
    _load().orc_conv3d_forward(_p(x), _p(w), _p(b), _p(y), _gp(g))
    return y


def conv3d_input_grad(dy, w, x_shape, stride=(1, 1, 1), pad=(0, 0, 0)):
    dy, w = _d(dy), _d(w)
    N, C, D, H, W = x_shape
    K, _, T, R, S = w.shape
    Do, P, Q = conv3d_out(D, H, W, T, R, S, stride, pad)
    g = _g3(N, C, D, H, W, K, T, R, S, Do, P, Q, stride, pad)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().orc_conv3d_input_grad(_p(dy), _p(w), _p(dx), _gp(g))
    return dx


def conv3d_weight_grad(dy, x, w_shape, stride=(1, 1, 1), pad=(0, 0, 0)):
    dy, x = _d(dy), _d(x)
    N, C, D, H, W = x.shape
    K, _, T, R, S = w_shape
    Do, P, Q = conv3d_out(D, H, W, T, R, S, stride, pad)
    g = _g3(N, C, D, H, W, K, T, R, S, Do, P, Q, stride, pad)
    dw = np.empty(tuple(w_shape), np.float64)
    _load().orc_conv3d_weight_grad(_p(dy), _p(x), _p(dw), _gp(g))
    return dw


def bias_grad5(dy):
    """db[k] = sum over (n, d, h, w) of dy[n, k, d, h, w]."""
    dy = _d(dy)
    N, K = dy.shape[:2]
    db = np.empty(K, np.float64)
    _load().orc_bias_grad5(_p(dy), _p(db), _I(N), _I(K), _I(int(np.prod(dy.shape[2:]))))
    return db


def convt3d_out(D, H, W, T, R, S, stride, pad, out_pad=(0, 0, 0)):
    if not all(0 <= o < s for o, s in zip(out_pad, stride)):
        raise ValueError("output padding must satisfy 0 <= out_pad < stride")
    out = tuple((e - 1) * s - 2 * p + k + o for e, k, s, p, o in zip((D, H, W), (T, R, S), stride, pad, out_pad))
    if min(out) < 1:
        raise ValueError("transposed convolution output would be empty")
    return out


def _convt3d_g(x_shape, w_shape, stride, pad, out_pad):
    N, Ci, D, H, W = x_shape
    Ci2, Co, T, R, S = w_shape
    if Ci2 != Ci:
        raise ValueError("channel mismatch")
    Do, Ho, Wo = convt3d_out(D, H, W, T, R, S, stride, pad, out_pad)
    return _g3(N, Ci, D, H, W, Co, T, R, S, Do, Ho, Wo, stride, pad), (N, Co, Do, Ho, Wo)


def convt3d_forward(x, w, b=None, stride=(1, 1, 1), pad=(0, 0, 0), out_pad=(0, 0, 0)):
    """Transposed 3-D convolution (torch.nn.ConvTranspose3d, App. B):
    x[N,Ci,D,H,W], W[Ci,Co,T,R,S], each input voxel scatters through each tap."""
    x, w, b = _d(x), _d(w), _d(b)
    g, ys = _convt3d_g(x.shape, w.shape, stride, pad, out_pad)
    y = np.empty(ys, np.float64)
    _load().orc_convt3d_forward(_p(x), _p(w), _p(b), _p(y), _gp(g))
    return y


def convt3d_input_grad(dy, w, x_shape, stride=(1, 1, 1), pad=(0, 0, 0), out_pad=(0, 0, 0)):
    dy, w = _d(dy), _d(w)
    g, _ = _convt3d_g(x_shape, w.shape, stride, pad, out_pad)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().orc_convt3d_input_grad(_p(dy), _p(w), _p(dx), _gp(g))
    return dx


def convt3d_weight_grad(dy, x, w_shape, stride=(1, 1, 1), pad=(0, 0, 0), out_pad=(0, 0, 0)):
    dy, x = _d(dy), _d(x)
    g, _ = _convt3d_g(x.shape, w_shape, stride, pad, out_pad)
    dw = np.empty(tuple(w_shape), np.float64)
    _load().orc_convt3d_weight_grad(_p(dy), _p(x), _p(dw), _gp(g))
    return dw
