"""Run-to-run bitwise determinism of the kernels that reduce without
atomics: split-K GEMMs and their reduce pass, the weight gradient's split
partials with the fused bias partials, the input gradient's fused column
sums and their finalize pass, the standalone column sum, the BN-eval
backward reduction, the fp32 path, the halo convolutions (stride phases,
k-group sums) and the 12-wave and paired Linear forwards.  Each reduction adds
its partials in a fixed order, so the same inputs give the same bytes on
every call."""
import os

import pytest
import torch

import paper_2404_12406_amd as ms
import synth

from _gpu import dev

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).clone()


def _twice(fn):
    a = [_bits(t) for t in fn() if t is not None]
    b = [_bits(t) for t in fn() if t is not None]
    assert len(a) == len(b) and len(a) > 0
    for i, (u, v) in enumerate(zip(a, b)):
        assert torch.equal(u, v), f"output {i} differs between two identical calls"


def _conv_case(xs, ws, stride, pad, dt, mask, seed):
    x = dev(synth.normal(xs, seed, dtype=dt), dt)
    w = dev(synth.kaiming_uniform(ws, seed + 1, ws[1] * ws[2] * ws[3], dtype=dt), dt)
    b = dev(synth.normal((ws[0],), seed + 2, 1.0, dtype=dt), dt)

    def run():
        y, rec = ms.layer_forward(ms.Conv2d(stride, pad), x, w, b, mask)
        gy = dev(synth.normal(tuple(y.shape), seed + 3, dtype=dt), dt)
        grads = ms.layer_backward(rec, gy) if rec is not None else ()
        torch.cuda.synchronize()
        return (y, *grads)
    return run


@pytest.fixture
def splits():
    old = os.environ.get("MEMSAVE_GEMM_SPLITS")
    os.environ["MEMSAVE_GEMM_SPLITS"] = "3"
    yield
    if old is None:
        del os.environ["MEMSAVE_GEMM_SPLITS"]
    else:
        os.environ["MEMSAVE_GEMM_SPLITS"] = old


def test_split_k_forward_and_input_gradient(splits):
    """Forward and input gradient with three reduction splits each: fp32
    partials summed by the reduce pass (which adds the forward bias)."""
    _twice(_conv_case((2, 64, 14, 13), (96, 64, 3, 3), (1, 1), (1, 1), "bf16", 7, 9900))


def test_weight_gradient_split_partials_and_fused_bias():
    """The 3x3 conv sweep's weight gradient (the planner splits its
    25088-long reduction) with the bias gradient fused into its partials."""
    _twice(_conv_case((32, 256, 28, 28), (256, 256, 3, 3), (1, 1), (1, 1), "bf16", 6, 9910))


def test_input_gradient_with_column_sums():
    """Mask input + bias of a Linear layer: the input-gradient blocks sum
    dy's columns into partial rows that the finalize pass adds in order."""
    x = dev(synth.normal((4096, 1024), 9920, dtype="bf16"), "bf16")
    w = dev(synth.normal((4096, 1024), 9921, 0.02, dtype="bf16"), "bf16")
    b = dev(synth.normal((4096,), 9922, 1.0, dtype="bf16"), "bf16")
    gy = dev(synth.normal((4096, 4096), 9923, dtype="bf16"), "bf16")

    def run():
        y, rec = ms.layer_forward(ms.Linear(), x, w, b, 5)
        gx, _, gb = ms.layer_backward(rec, gy)
        torch.cuda.synchronize()
        return y, gx, gb
    _twice(run)


def test_standalone_column_sum():
    """A bias-only mask: the backward is the column sum of dy alone."""
    _twice(_conv_case((8, 64, 28, 28), (64, 64, 3, 3), (1, 1), (1, 1), "bf16", 4, 9930))


@pytest.mark.parametrize("mask", [1, 2, 4, 7])
def test_bn_eval_backward_reduction(mask):
    shape = (16, 64, 28, 28)
    C = shape[1]
    x = dev(synth.normal(shape, 9940, dtype="bf16"), "bf16")
    mu = dev(synth.normal((C,), 9941, 0.1, dtype="bf16"), "bf16")
    var = dev(synth.uniform((C,), 9942, 0.5, 1.5, dtype="bf16"), "bf16")
    g = dev(synth.uniform((C,), 9943, 0.5, 1.5, dtype="bf16"), "bf16")
    be = dev(synth.normal((C,), 9944, 0.1, dtype="bf16"), "bf16")
    gy = dev(synth.normal(shape, 9945, dtype="bf16"), "bf16")

    def run():
        y, rec = ms.layer_forward(ms.BatchNormEval(mu, var, 1e-5), x, g, be, mask)
        grads = ms.layer_backward(rec, gy)
        torch.cuda.synchronize()
        return (y, *grads)
    _twice(run)


def test_fp32_path_with_splits():
    """The fp32 kernels (and their split-K reduce) on the fp32 single-conv
    shape with every flag."""
    _twice(_conv_case((8, 16, 32, 32), (32, 16, 3, 3), (1, 1), (1, 1), "f32", 7, 9950))


@pytest.mark.parametrize("case", [
    ((2, 64, 23, 21), (64, 64, 3, 3), (2, 2), (1, 1)),   # halo: stride-2 input phases and output phases
    ((2, 64, 13, 11), (64, 64, 3, 3), (1, 1), (1, 1)),   # halo: the unrolled 3x3 schedule, both ways
    ((2, 3, 30, 32), (64, 3, 7, 7), (2, 2), (3, 3)),     # stem blocks: 16-channel forward, two-k-group input gradient
])
def test_halo_convolutions(case):
    """The halo kernels accumulate taps and stride phases in a fixed order
    (the two-k-group form adds group 1's sums through LDS): every output and
    gradient repeats byte for byte."""
    xs, ws, stride, pad = case
    _twice(_conv_case(xs, ws, stride, pad, "bf16", 7, 9960))


@pytest.mark.parametrize("n_out", [2304, 3072])
def test_twelve_wave_and_paired_linear_forward(n_out):
    """8192-row Linear forwards on the 256 x 288 tile (2304 outputs, one
    wave) and on the paired column split (3072 outputs: 256 x 256 then
    256 x 128 tiles in one launch), with the input gradient of each."""
    M, Kin = 8192, 136
    x = dev(synth.normal((M, Kin), 9970, dtype="bf16"), "bf16")
    w = dev(synth.normal((n_out, Kin), 9971, 0.05, dtype="bf16"), "bf16")
    b = dev(synth.normal((n_out,), 9972, 1.0, dtype="bf16"), "bf16")
    gy = dev(synth.normal((M, n_out), 9973, dtype="bf16"), "bf16")

    def run():
        y, rec = ms.layer_forward(ms.Linear(), x, w, b, 1)
        grads = ms.layer_backward(rec, gy)
        torch.cuda.synchronize()
        return (y, *grads)
    _twice(run)
