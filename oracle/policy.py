"""Closed-form save rule and retained-byte accounting (TEST INFRASTRUCTURE).

The rule (Sec. 2.2.1): for a layer Z = W * X + b that is linear in X and in
W, the input Jacobian needs W, the weight Jacobian needs X and the bias
Jacobian needs nothing; the layer checks which of W, X (and b) require grad
and stores only what the Jacobians that will be applied need.  The same holds
for batch normalisation in evaluation mode with gamma in the role of W:
the input gradient needs gamma and sigma_hat^2, the gamma gradient needs x,
mu_hat and sigma_hat^2 (App. C).  The transposed convolution is linear in x
and in W as well (Sec. 2.2.1 names it beside the convolution) and follows the
convolution's rule.

Comparison policies:
  SELECTIVE        the rule above;
  PYTORCH_DEFAULT  what stock PyTorch saves under the same mask: convolution,
                   its transpose and BN-eval store their input whenever the node exists,
                   i.e. whenever any parent requires grad (Fig. 2, Sec. 2.1,
                   App. B); the fully-connected layer is already agnostic
                   (App. B), so it follows SELECTIVE;
  ALL_TRUE         every parent requires grad ("All" case of Sec. 3).

Only non-parameter tensors count as retained activation bytes; parameters
and running statistics are resident anyway and are reported separately.
A mask of 0 creates no record at all (no node is recorded).

ReLU (Sec. 2.2.2): stock PyTorch keeps the output, which may be the next
linear layer's input; the paper's ReLU keeps a boolean mask of the output
instead, one byte per element, and this library one bit per element (4-byte
words: 4 * ceil(n / 32) bytes).  It has no parameters, so ALL_TRUE is its
INPUT mask.

Dropout (Sec. 2.2.2): stock PyTorch keeps its one-byte boolean mask; the
paper's dropout, and this library's, keeps the random state and draws the
mask again in backward, so it keeps no activation bytes.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

MASK_INPUT, MASK_WEIGHT, MASK_BIAS = 1, 2, 4
SELECTIVE, PYTORCH_DEFAULT, ALL_TRUE = 0, 1, 2
ELT = {"f32": 4, "bf16": 2}


def saved_tensors(kind: str, mask: int, policy: int = SELECTIVE,
                  has_weight: bool = True, has_bias: bool = True) -> Dict[str, bool]:
    """Which tensors a layer of `kind` keeps for backward under `mask`.

    Returns a dict with keys 'x' (the layer input, an activation) and the
    parameter-side references ('W' for conv/linear; 'gamma', 'running_mean',
    'running_var' for BN-eval)."""
    if policy == ALL_TRUE:
        mask = MASK_INPUT | (MASK_WEIGHT if has_weight else 0) | (MASK_BIAS if has_bias else 0)
    i = bool(mask & MASK_INPUT)
    w = bool(mask & MASK_WEIGHT)
    any_flag = mask != 0
    if kind in ("conv2d", "conv_transpose2d", "conv3d", "conv_transpose3d", "linear"):
        if policy == PYTORCH_DEFAULT and kind != "linear":
            return {"x": any_flag, "W": any_flag}
        return {"x": w, "W": i}
    if kind == "bn_eval":
        if policy == PYTORCH_DEFAULT:
            return {"x": any_flag, "gamma": any_flag and has_weight,
                    "running_mean": any_flag, "running_var": any_flag}
        return {"x": w, "gamma": i and has_weight, "running_mean": w,
                "running_var": i or w}
    if kind == "avgpool":
        return {"x": False}
    if kind == "relu":
        if policy == PYTORCH_DEFAULT:
            return {"x": False, "y": i, "bits": False}
        return {"x": False, "y": False, "bits": i}
    if kind == "dropout":
        # stock PyTorch keeps a one-byte boolean mask; this library the
        # generator's key and counter (no device memory)
        return {"x": False, "mask8": i and policy == PYTORCH_DEFAULT, "rng_state": i and policy != PYTORCH_DEFAULT}
    raise ValueError(kind)


def relu_mask_bytes(numel: int) -> int:
    """Bytes of a ReLU record's 1-bit mask."""
    return 4 * ((int(numel) + 31) // 32) if numel > 0 else 0


def saved_activation_bytes(kind: str, mask: int, x_numel: int, dtype: str,
                           policy: int = SELECTIVE, has_weight: bool = True,
                           has_bias: bool = True) -> int:
    st = saved_tensors(kind, mask, policy, has_weight, has_bias)
    if kind == "relu":
        if st["y"]:
            return int(x_numel) * ELT[dtype]
        return relu_mask_bytes(x_numel) if st["bits"] else 0
    if kind == "dropout":
        return int(x_numel) if st["mask8"] else 0
    return int(x_numel) * ELT[dtype] if st["x"] else 0


def launched(kind: str, mask: int) -> Dict[str, bool]:
    """Backward launch plan: the input-, weight- and bias-gradient work runs
    exactly when its flag is set (Sec. 2.2.1)."""
    if kind in ("avgpool", "relu", "dropout"):
        return {"dgrad": bool(mask & MASK_INPUT), "wgrad": False, "bgrad": False}
    return {"dgrad": bool(mask & MASK_INPUT), "wgrad": bool(mask & MASK_WEIGHT),
            "bgrad": bool(mask & MASK_BIAS)}


def propagate(param_flags: Sequence[int], input_requires_grad: bool) -> List[int]:
    """Masks of a chain of layers from their parameter flags (bits 2 and 4)
    and whether the chain's input requires grad: a layer output requires grad
    as soon as any of its parents does (Sec. 2), so layer l's input bit is set
    iff the chain input or any parameter of an earlier layer requires grad."""
    out = []
    rg = bool(input_requires_grad)
    for f in param_flags:
        f = int(f) & (MASK_WEIGHT | MASK_BIAS)
        m = f | (MASK_INPUT if rg else 0)
        out.append(m)
        rg = rg or f != 0
    return out


def stack_saved_bytes(layers, policy: int = SELECTIVE) -> int:
    """Total retained activation bytes of a stack at the end of its forward
    pass: the sum over every layer's record.  `layers` is an iterable of
    (kind, mask, x_numel, dtype[, has_weight, has_bias]) tuples."""
    tot = 0
    for t in layers:
        kind, mask, numel, dtype = t[:4]
        hw = t[4] if len(t) > 4 else True
        hb = t[5] if len(t) > 5 else True
        if mask == 0 and policy != ALL_TRUE:
            continue
        tot += saved_activation_bytes(kind, mask, numel, dtype, policy, hw, hb)
    return tot
