"""Pins of the closed-form save rule against the paper's statements:
the Fig. 2 truth table, the 512 MiB-per-layer slope and the layer-4
experiment of Sec. 2.1, App. B (Linear already agnostic) and App. C (BN-eval
input gradient needs no input), and the per-workload totals."""
import json
import os

import pytest

from oracle import policy as P
from synth import workloads as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _stores(kind, mask, pol):
    st = P.saved_tensors(kind, mask, pol)
    return sorted(k.replace("x", "X") for k, v in st.items() if v)


def test_fig2_truth_table():
    g = json.load(open(os.path.join(GOLD, "fig2_truth_table.json")))
    for row in g["rows"]:
        mask = (P.MASK_WEIGHT if row["W_rg"] else 0) | (P.MASK_INPUT if row["X_rg"] else 0)
        assert _stores("conv2d", mask, P.PYTORCH_DEFAULT) == sorted(row["pytorch"]), row
        assert _stores("conv2d", mask, P.SELECTIVE) == sorted(row["memsave"]), row


def _e1_stack(depth, case):
    """Masks of the synthetic CNN of Sec. 2.1 (input never requires grad)."""
    if case == "all":
        flags = [P.MASK_WEIGHT] * depth
    elif case == "none":
        flags = [0] * depth
    elif case == "4plus":
        flags = [0 if l < 3 else P.MASK_WEIGHT for l in range(depth)]
    elif case == "only4":
        flags = [P.MASK_WEIGHT if l == 3 else 0 for l in range(depth)]
    return P.propagate(flags, False)


@pytest.mark.parametrize("case", ["all", "none", "4plus", "only4"])
def test_e1_synthetic_cnn(case):
    g = json.load(open(os.path.join(GOLD, "e1_synthetic_cnn.json")))
    n, c, h, w = g["x_shape"]
    numel = n * c * h * w
    per = g["bytes_per_stored_input"]
    assert numel * 4 == per == 512 * 2**20
    for depth in g["depths"]:
        masks = _e1_stack(depth, case)
        layers = [("conv2d", m, numel, "f32", True, False) for m in masks]
        sel = P.stack_saved_bytes(layers, P.SELECTIVE)
        pt = P.stack_saved_bytes(layers, P.PYTORCH_DEFAULT)
        after3 = max(0, depth - 3)
        if case == "all":
            assert sel == pt == depth * per                  # slope 512 MiB per layer
        elif case == "none":
            assert sel == pt == 0
        elif case == "4plus":
            assert sel == pt == after3 * per
        elif case == "only4":
            assert pt == after3 * per                         # same as layers 4+ for PyTorch
            assert sel == (per if depth >= 4 else 0)          # only layer 4's input


def test_linear_already_agnostic_and_bn_eval_rule():
    for mask in range(8):
        assert P.saved_tensors("linear", mask, P.PYTORCH_DEFAULT) == P.saved_tensors("linear", mask, P.SELECTIVE)
    # BN eval, input-only: PyTorch keeps x, the rule does not (App. C)
    assert P.saved_tensors("bn_eval", P.MASK_INPUT, P.PYTORCH_DEFAULT)["x"]
    assert not P.saved_tensors("bn_eval", P.MASK_INPUT, P.SELECTIVE)["x"]
    assert P.saved_tensors("bn_eval", P.MASK_WEIGHT, P.SELECTIVE)["x"]
    for kind in ("conv2d", "linear", "bn_eval"):
        for mask in range(8):
            assert P.saved_tensors(kind, mask, P.SELECTIVE)["x"] == bool(mask & P.MASK_WEIGHT)
            plan = P.launched(kind, mask)
            assert plan == {"dgrad": bool(mask & 1), "wgrad": bool(mask & 2), "bgrad": bool(mask & 4)}


def test_propagation_rule():
    assert P.propagate([0, 0, 0], False) == [0, 0, 0]
    assert P.propagate([0, 0, 0], True) == [1, 1, 1]
    assert P.propagate([0, 6, 0, 0], False) == [0, 6, 1, 1]
    assert P.propagate([4, 0], False) == [4, 1]


def _workload_bytes(w, policy):
    layers = []
    for l in w.layers:
        numel = 1
        for s in l.in_shape:
            numel *= s
        layers.append((l.kind, l.mask, numel, w.dtype, l.kind != "avgpool", l.has_bias))
    return P.stack_saved_bytes(layers, policy)


def test_workload_retained_bytes():
    """Totals of the five synthetic workloads (selective / PyTorch / all-true)."""
    exp = {
        "1": (0, 524288, 524288),
        "2": (0, 0, 83886080),
        "3": (65536, 65536, 606994432),
        "3b": (606994432 - 65536 + 65536, 606994432, 606994432),
        "5": (0, 0, 1056964608),
        "4_3x3_00": (0, 0, 12845056), "4_3x3_10": (0, 12845056, 12845056),
        "4_3x3_01": (12845056, 12845056, 12845056), "4_3x3_11": (12845056, 12845056, 12845056),
        "4_1x1_10": (0, 12845056, 12845056),
    }
    ws = wl.all_workloads()
    for name, (sel, pt, allt) in exp.items():
        w = ws[name]
        got = tuple(_workload_bytes(w, p) for p in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE))
        if name == "3b":
            # 'Input' variant: convs/BN keep nothing (frozen), the Linear keeps its input
            assert got[0] == 65536 and got[1] == 606994432 and got[2] == 606994432
            continue
        assert got == (sel, pt, allt), (name, got)


def test_workload_masks_follow_propagation():
    ws = wl.all_workloads()
    for name in ("3", "3b"):
        w = ws[name]
        flags = [l.mask & 6 for l in w.layers]
        assert [l.mask for l in w.layers] == P.propagate(flags, name == "3b")
