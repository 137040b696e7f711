"""A chain of layers run through the C ABI: forward in order, backward in
reverse, with every activation and gradient buffer allocated once.

Each layer's mask is given by the caller (a layer's input requires grad
when the chain input or any earlier parameter does, Sec. 2).  Backward
feeds layer l+1's input gradient to layer l as its output gradient; layers
with mask 0 record nothing and are skipped."""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import torch

from .api import BatchNormEval, PreparedLayer, empty_like_layout, output_shape


@dataclass
class LayerCall:
    spec: object
    W: Optional[torch.Tensor] = None
    b: Optional[torch.Tensor] = None
    mask: int = 0


class Chain:
    def __init__(self, layers: List[LayerCall], x: torch.Tensor, grad_y: Optional[torch.Tensor] = None):
        self.calls = layers
        self.acts = [x]
        for lc in layers:
            self.acts.append(empty_like_layout(output_shape(lc.spec, self.acts[-1], lc.W), x))
        self.grad_y = grad_y
        self.grads = []
        gx_next = grad_y
        prepared = [None] * len(layers)
        grads = [None] * len(layers)
        for i in range(len(layers) - 1, -1, -1):
            lc = layers[i]
            xin = self.acts[i]
            gx = empty_like_layout(tuple(xin.shape), xin) if lc.mask & 1 else None
            gw = empty_like_layout(tuple(lc.W.shape), lc.W) if lc.mask & 2 else None
            gb = torch.empty_like(lc.b) if lc.mask & 4 else None
            gy = gx_next if lc.mask else None
            if lc.mask and gy is None:
                raise ValueError(f"layer {i} needs an output gradient but the next layer does not pass one")
            prepared[i] = PreparedLayer(lc.spec, xin, lc.W, lc.b, lc.mask, self.acts[i + 1],
                                        gy, gx, gw, gb)
            grads[i] = (gx, gw, gb)
            gx_next = gx
        self.prepared = prepared
        self.grads = grads

    @property
    def y(self) -> torch.Tensor:
        return self.acts[-1]

    def forward(self):
        for p in self.prepared:
            p.forward()

    def backward(self):
        for p in reversed(self.prepared):
            if p.mask:
                p.backward()
