"""Place drawn workload arrays on the GPU and wire them into the library's
Chain executor (imported only by the benchmark and the GPU tests).  Values
are copied exactly: the arrays are already rounded to the workload dtype."""
from __future__ import annotations

from typing import List

import numpy as np
import torch

import paper_2404_12406_amd as ms
from paper_2404_12406_amd.stack import Chain, LayerCall

from .draw import ChainArrays

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def dev(a, dtype: str, device="cuda"):
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_DT[dtype])
    if t.dim() == 4:
        t = t.contiguous(memory_format=torch.channels_last)
    return t.to(device)


def layer_call(la, dtype: str) -> LayerCall:
    s = la.spec
    if s.kind == "conv2d":
        spec = ms.Conv2d(s.stride, s.pad)
    elif s.kind == "conv_transpose2d":
        spec = ms.ConvTranspose2d(s.stride, s.pad, s.out_pad)
    elif s.kind == "linear":
        spec = ms.Linear()
    elif s.kind == "bn_eval":
        spec = ms.BatchNormEval(dev(la.running_mean, dtype), dev(la.running_var, dtype), s.eps)
    elif s.kind == "avgpool":
        spec = ms.AvgPool()
    else:
        raise ValueError(s.kind)
    return LayerCall(spec, dev(la.W, dtype), dev(la.b, dtype), s.mask)


def build_chain(ca: ChainArrays, dtype: str, with_grad: bool = True) -> Chain:
    calls = [layer_call(la, dtype) for la in ca.layers]
    return Chain(calls, dev(ca.x, dtype), dev(ca.grad_y, dtype) if with_grad else None)


def build_chains(chains: List[ChainArrays], dtype: str) -> List[Chain]:
    return [build_chain(c, dtype) for c in chains]
