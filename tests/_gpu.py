"""Helpers for the GPU parity tests: move seeded host arrays to the device in
the layout the library needs, bring results back as float64 in logical
order, and the tolerance bar (normwise max relative error).  Nothing here
computes a layer."""
from __future__ import annotations

import numpy as np
import torch

import oracle

TOL = {"f32": 1e-4, "bf16": 2e-2}
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 host array (already rounded to `dtype`) -> device tensor;
    4-D tensors are stored channels-last."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_DT[dtype])
    if t.dim() == 4:
        t = t.contiguous(memory_format=torch.channels_last)
    return t.cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


# (test id, output name, observed error, bar) of every check, for the
# session's margin report (tests/conftest.py)
MARGINS = []


def check(name, got, ref, dtype, tol=None):
    """Normwise relative error of `got` against the oracle's `ref` (both in
    logical order), asserted against the bar; the observed error is logged."""
    import os
    tol = TOL[dtype] if tol is None else tol
    err = oracle.rel_err(got, ref)
    MARGINS.append((os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0], name, err, tol))
    print(f"[parity] {name}: normwise rel err {err:.3e} (bar {tol:.0e})")
    assert err <= tol, f"{name}: normwise rel err {err:.3e} > {tol:.0e}"
    return err


def guarded_empty(shape, dtype: str, guard: int = 64, fill=float("nan")):
    """An output tensor (channels-last for 4-D) living in the middle of a
    larger buffer whose guard bands hold `fill`; returns (view, buffer, guard)."""
    numel = int(np.prod(shape)) if len(shape) else 1
    buf = torch.full((numel + 2 * guard,), fill, dtype=TORCH_DT[dtype], device="cuda")
    if len(shape) == 4:
        N, C, H, W = shape
        strides = (H * W * C, 1, W * C, C)
    elif len(shape) == 2:
        strides = (shape[1], 1)
    else:
        strides = (1,)
    view = buf.as_strided(shape, strides, guard)
    return view, buf, guard


def guards_intact(buf: torch.Tensor, guard: int, fill=float("nan")) -> bool:
    g = torch.cat([buf[:guard], buf[-guard:]]).float().cpu()
    if np.isnan(fill):
        return bool(torch.isnan(g).all())
    return bool((g == fill).all())
