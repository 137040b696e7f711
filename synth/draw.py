"""Draw the host arrays of a workload (seeded; float32 values rounded to the
workload dtype).  A workload is a list of layers; a layer whose input is not
chained starts a new chain that gets its own input, and every chain gets its
own output gradient.  No layer arithmetic happens here."""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import kaiming_uniform, normal, uniform
from .workloads import LayerSpec, Workload


@dataclass
class LayerArrays:
    spec: LayerSpec
    W: Optional[np.ndarray] = None
    b: Optional[np.ndarray] = None
    running_mean: Optional[np.ndarray] = None
    running_var: Optional[np.ndarray] = None


@dataclass
class ChainArrays:
    layers: List[LayerArrays]
    x: np.ndarray
    grad_y: np.ndarray
    x_requires_grad: bool = False


def _draw(law, shape, seed, dtype):
    kind, params = law
    if kind == "normal":
        return normal(shape, seed, std=params[1], mean=params[0], dtype=dtype)
    if kind == "uniform":
        return uniform(shape, seed, params[0], params[1], dtype=dtype)
    if kind == "kaiming":
        return kaiming_uniform(shape, seed, params[0], dtype=dtype)
    raise ValueError(kind)


def layer_arrays(spec: LayerSpec, dtype: str) -> LayerArrays:
    la = LayerArrays(spec)
    ws = spec.weight_shape()
    if "W" in spec.init and ws is not None:
        la.W = _draw(spec.init["W"], ws, spec.seeds["W"], dtype)
    if spec.has_bias and "b" in spec.init:
        n = spec.in_shape[1] if spec.kind == "bn_eval" else spec.out_ch
        la.b = _draw(spec.init["b"], (n,), spec.seeds["b"], dtype)
    if spec.kind == "bn_eval":
        C = spec.in_shape[1]
        la.running_mean = _draw(spec.init["running_mean"], (C,), spec.seeds["running_mean"], dtype)
        la.running_var = _draw(spec.init["running_var"], (C,), spec.seeds["running_var"], dtype)
    return la


def chains(w: Workload) -> List[ChainArrays]:
    """Split a workload into chains and draw every array."""
    groups: List[List[LayerSpec]] = []
    for spec in w.layers:
        if not groups or not spec.chained_input:
            groups.append([])
        groups[-1].append(spec)
    out = []
    base = 1000 * w.index + 500
    for ci, g in enumerate(groups):
        first = g[0]
        x_seed = first.seeds.get("x", w.input_seed)
        x = _draw(w.input_law, first.in_shape, x_seed, w.dtype)
        gy = _draw(w.grad_law, g[-1].out_shape(), base + ci, w.dtype)
        out.append(ChainArrays([layer_arrays(s, w.dtype) for s in g], x, gy,
                               bool(first.mask & 1)))
    return out
