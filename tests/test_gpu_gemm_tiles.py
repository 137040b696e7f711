"""Every tile shape of the bf16 implicit-GEMM fast path, forced through
MEMSAVE_GEMM_TILE, in all three contractions and both input-gradient variants, on ragged sizes (including a
strided input gradient and a fused bias gradient), against the oracle."""
import os

import numpy as np
import torch
import pytest

import oracle
import paper_2404_12406_amd as ms
import synth

from _gpu import check, dev, host

pytestmark = pytest.mark.gpu

# biases are drawn at the outputs' scale (N(0, 1)), so a dropped or
# misplaced bias fails the 2e-2 bar by far
TILES = ["256x256", "256x128", "128x128", "128x128w8", "128x128s4", "128x128w8s4", "128x128k2", "128x64", "256x32",
         "128x192k2", "256x288"]

CASES = [
    # x shape, w shape, stride, pad
    ((3, 24, 13, 11), (40, 24, 3, 3), (1, 1), (1, 1)),
    ((2, 16, 15, 14), (24, 16, 3, 3), (2, 2), (1, 1)),
    ((2, 64, 9, 10), (136, 64, 1, 1), (1, 1), (0, 0)),
    ((1, 48, 12, 9), (72, 48, 5, 3), (3, 2), (2, 1)),
    ((2, 80, 20, 18), (264, 80, 3, 3), (1, 1), (1, 1)),   # several 256-wide tiles, ragged in M, N and k
    ((2, 3, 30, 29), (16, 3, 7, 7), (2, 2), (3, 3)),      # 3 channels: zero-padded to 8 for the fast path
    ((1, 12, 20, 18), (24, 12, 3, 3), (1, 1), (1, 1)),    # 12 channels: padded to 16
]


@pytest.fixture(params=["transposed", "direct"])
def dgrad_variant(request):
    """Both input-gradient variants: through a transposed copy of W, and
    reading W in place (MEMSAVE_DGRAD)."""
    old = os.environ.get("MEMSAVE_DGRAD")
    os.environ["MEMSAVE_DGRAD"] = request.param
    yield request.param
    if old is None:
        del os.environ["MEMSAVE_DGRAD"]
    else:
        os.environ["MEMSAVE_DGRAD"] = old


@pytest.fixture
def tile(request):
    old = os.environ.get("MEMSAVE_GEMM_TILE")
    os.environ["MEMSAVE_GEMM_TILE"] = request.param
    yield request.param
    if old is None:
        del os.environ["MEMSAVE_GEMM_TILE"]
    else:
        os.environ["MEMSAVE_GEMM_TILE"] = old


@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("case", range(len(CASES)))
def test_conv_tiles(tile, case, dgrad_variant):
    xs, ws, stride, pad = CASES[case]
    seed = 7000 + 10 * case
    x = synth.normal(xs, seed, dtype="bf16")
    w = synth.kaiming_uniform(ws, seed + 1, ws[1] * ws[2] * ws[3], dtype="bf16")
    b = synth.normal((ws[0],), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    check("y", host(y), oracle.conv2d_forward(x, w, b, stride, pad), "bf16")
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(gx), oracle.conv2d_input_grad(gy, w, xs, stride, pad), "bf16")
    check("dW", host(gw), oracle.conv2d_weight_grad(gy, x, ws, stride, pad), "bf16")
    check("db", host(gb), oracle.conv2d_bias_grad(gy), "bf16")


@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("shape", [(300, 72, 136), (520, 264, 392), (1000, 520, 64)])
def test_linear_tiles(tile, shape, dgrad_variant):
    M, Kin, Nout = shape
    seed = 7500 + M
    x = synth.normal((M, Kin), seed, dtype="bf16")
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype="bf16")
    b = synth.normal((Nout,), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Linear(), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    y_ref = oracle.linear_forward(x, w, b)
    assert oracle.rel_err(oracle.linear_forward(x, w, None), y_ref) > 0.2   # the bias is visible at the bar
    check("y", host(y), y_ref, "bf16")
    gy = synth.normal((M, Nout), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dX", host(gx), oracle.linear_input_grad(gy, w), "bf16")
    check("dW", host(gw), oracle.linear_weight_grad(gy, x), "bf16")
    check("db", host(gb), oracle.linear_bias_grad(gy), "bf16")


@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("shape", [(300, 72, 136), (520, 264, 392), (1000, 520, 64), (4100, 64, 1032),
                                   (300, 72, 4200), (700, 1032, 40)])
def test_linear_tiles_bias_without_weight_gradient(tile, shape, dgrad_variant):
    """Mask input + bias (weight frozen, the fine-tuning mask): the input
    gradient on every tile, the bias gradient taken along by its blocks
    (dy's columns shared out over the block columns; several 512-column
    passes when the output is narrow, block columns with no share when it is
    wide), with rows ragged against every block height and reductions ragged
    against the 64-deep step."""
    M, Kin, Nout = shape
    seed = 7700 + M
    x = synth.normal((M, Kin), seed, dtype="bf16")
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype="bf16")
    b = synth.normal((Nout,), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Linear(), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 5)
    gy = synth.normal((M, Nout), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    assert gw is None
    check("dX", host(gx), oracle.linear_input_grad(gy, w), "bf16")
    check("db", host(gb), oracle.linear_bias_grad(gy), "bf16")


@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("case", range(len(CASES)))
def test_conv_tiles_bias_without_weight_gradient(tile, case, dgrad_variant):
    """Mask input + bias on every conv case and tile."""
    xs, ws, stride, pad = CASES[case]
    seed = 7800 + 10 * case
    x = synth.normal(xs, seed, dtype="bf16")
    w = synth.kaiming_uniform(ws, seed + 1, ws[1] * ws[2] * ws[3], dtype="bf16")
    b = synth.normal((ws[0],), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 5)
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    assert gw is None
    check("dx", host(gx), oracle.conv2d_input_grad(gy, w, xs, stride, pad), "bf16")
    check("db", host(gb), oracle.conv2d_bias_grad(gy), "bf16")


@pytest.fixture
def splits(request):
    """Force the split count of the forward and input-gradient GEMMs
    (MEMSAVE_GEMM_SPLITS): fp32 partials summed by a second pass, the
    forward bias added there."""
    old = os.environ.get("MEMSAVE_GEMM_SPLITS")
    os.environ["MEMSAVE_GEMM_SPLITS"] = request.param
    yield request.param
    if old is None:
        del os.environ["MEMSAVE_GEMM_SPLITS"]
    else:
        os.environ["MEMSAVE_GEMM_SPLITS"] = old


@pytest.mark.parametrize("splits", ["3"], indirect=True)
@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("case", range(len(CASES)))
def test_conv_tiles_split(tile, case, splits):
    """Split reductions on every conv case and tile: strided input
    gradients put each phase's partial rows at their own dx pixels, and
    splits past a short reduction contribute zeros."""
    xs, ws, stride, pad = CASES[case]
    seed = 7900 + 10 * case
    x = synth.normal(xs, seed, dtype="bf16")
    w = synth.kaiming_uniform(ws, seed + 1, ws[1] * ws[2] * ws[3], dtype="bf16")
    b = synth.normal((ws[0],), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    check("y", host(y), oracle.conv2d_forward(x, w, b, stride, pad), "bf16")
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(gx), oracle.conv2d_input_grad(gy, w, xs, stride, pad), "bf16")
    check("dW", host(gw), oracle.conv2d_weight_grad(gy, x, ws, stride, pad), "bf16")
    check("db", host(gb), oracle.conv2d_bias_grad(gy), "bf16")


@pytest.mark.parametrize("splits", ["2", "5"], indirect=True)
@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("shape", [(300, 72, 136), (520, 264, 392), (1000, 520, 64), (300, 72, 138)])
def test_linear_tiles_split(tile, shape, splits):
    """Split reductions of the Linear forward (bias added by the reduce) and
    input gradient; N_out = 138 leaves rows of partials that are not whole
    16-byte vectors (the input gradient then takes the general kernel)."""
    M, Kin, Nout = shape
    seed = 7600 + M + Nout
    x = synth.normal((M, Kin), seed, dtype="bf16")
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype="bf16")
    b = synth.normal((Nout,), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Linear(), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 5)
    check("y", host(y), oracle.linear_forward(x, w, b), "bf16")
    gy = synth.normal((M, Nout), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    assert gw is None
    check("dX", host(gx), oracle.linear_input_grad(gy, w), "bf16")
    check("db", host(gb), oracle.linear_bias_grad(gy), "bf16")


CONVT_CASES = [
    # x shape, C_out, (R, S), stride, pad, out_pad
    ((2, 24, 7, 6), 40, (4, 4), (2, 2), (1, 1), (1, 0)),
    ((2, 64, 5, 5), 264, (3, 3), (1, 1), (1, 1), (0, 0)),    # several 256-wide tiles, ragged
    ((1, 16, 9, 8), 12, (2, 2), (2, 2), (0, 0), (0, 0)),     # 12 output channels: padded, bias padded
]


def _convt_case(case, seed):
    xs, co, k, st, pd, op = CONVT_CASES[case]
    ws = (xs[1], co, k[0], k[1])
    x = synth.normal(xs, seed, dtype="bf16")
    w = synth.kaiming_uniform(ws, seed + 1, co * k[0] * k[1], dtype="bf16")
    b = synth.normal((co,), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.ConvTranspose2d(st, pd, op), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    check("y", host(y), oracle.convt2d_forward(x, w, b, st, pd, op), "bf16")
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(gx), oracle.convt2d_input_grad(gy, w, xs, st, pd, op), "bf16")
    check("dW", host(gw), oracle.convt2d_weight_grad(gy, x, ws, st, pd, op), "bf16")
    check("db", host(gb), oracle.convt2d_bias_grad(gy), "bf16")


@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("case", range(len(CONVT_CASES)))
def test_conv_transpose_tiles(tile, case, dgrad_variant):
    """The transposed convolution on every tile and input-gradient variant:
    its forward is the input-gradient contraction with the bias added in the
    epilogue, its input gradient the forward contraction."""
    _convt_case(case, 8800 + 10 * case)


@pytest.mark.parametrize("splits", ["3"], indirect=True)
@pytest.mark.parametrize("tile", TILES, indirect=True)
@pytest.mark.parametrize("case", range(len(CONVT_CASES)))
def test_conv_transpose_tiles_split(tile, case, splits):
    """Split reductions: the bias is added once, by the reduce pass."""
    _convt_case(case, 8900 + 10 * case)


@pytest.fixture
def tail_split():
    """Take the column split wherever it applies (MEMSAVE_GEMM_TAIL=on): the
    output's leading tile columns that fill whole waves of 256 CUs in one
    launch, the rest with another tile in a second launch."""
    old = os.environ.get("MEMSAVE_GEMM_TAIL")
    os.environ["MEMSAVE_GEMM_TAIL"] = "on"
    yield
    if old is None:
        del os.environ["MEMSAVE_GEMM_TAIL"]
    else:
        os.environ["MEMSAVE_GEMM_TAIL"] = old


@pytest.mark.parametrize("shape", [(8200, 136, 2312), (8192, 64, 3072), (8192, 72, 2304),
                                   (8200, 2312, 136), (8192, 3072, 64), (8192, 2304, 72)])
def test_linear_column_split(shape, dgrad_variant, tail_split):
    """Outputs of more than one wave of 256 x 256 tiles with a partial last
    wave: the forward (wide N_out; the bias added past the split column) and
    the input gradient (wide K_in; W read in place, or through the transposed
    copy), with remainders on the 256 x 128, 128 x 128 k-group and 128 x 192
    tiles, one row from every 64-row band and the last rows, every column."""
    M, Kin, Nout = shape
    seed = 7300 + M + Nout
    x = synth.normal((M, Kin), seed, dtype="bf16")
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype="bf16")
    b = synth.normal((Nout,), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Linear(), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 1)
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([np.arange(0, M, 64) + rng.integers(0, 64, (M + 63) // 64), [M - 2, M - 1]]))
    rows = rows[rows < M]
    yr = oracle.linear_forward(x[rows], w, b)
    assert oracle.rel_err(oracle.linear_forward(x[rows], w, None), yr) > 0.2
    check("y", host(y)[rows], yr, "bf16")
    gy = synth.normal((M, Nout), seed + 3, dtype="bf16")
    (gx,) = [g for g in ms.layer_backward(rec, dev(gy, "bf16")) if g is not None]
    check("dX", host(gx)[rows], oracle.linear_input_grad(gy[rows], w), "bf16")


@pytest.mark.parametrize("variant", ["forward", "transposed", "direct"])
def test_paired_column_split_matches_two_launches(variant, monkeypatch):
    """An 8192 x 3072 output is a column split of 256 tiles of 256 x 256 and
    256 tiles of 256 x 128: one paired launch by default, two launches with
    MEMSAVE_GEMM_PAIR=off.  Same tiles and reduction order, so the outputs
    agree byte for byte: the forward (its bias added past the split column),
    and the input gradient through the transposed copy and reading W in
    place.  The reductions (136 deep) end inside a 64-deep step."""
    M, K = 8192, 136
    Kin, Nout = (K, 3072) if variant == "forward" else (3072, K)
    seed = 7900 + len(variant)
    x = synth.normal((M, Kin), seed, dtype="bf16")
    w = synth.normal((Nout, Kin), seed + 1, 0.05, dtype="bf16")
    b = synth.normal((Nout,), seed + 2, 1.0, dtype="bf16")
    gy = synth.normal((M, Nout), seed + 3, dtype="bf16")
    if variant != "forward":
        monkeypatch.setenv("MEMSAVE_DGRAD", variant)
    outs = []
    for pair in ("on", "off"):
        monkeypatch.setenv("MEMSAVE_GEMM_PAIR", pair)
        y, rec = ms.layer_forward(ms.Linear(), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 1)
        (gx,) = [g for g in ms.layer_backward(rec, dev(gy, "bf16")) if g is not None]
        outs.append(y if variant == "forward" else gx)
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    rows = np.array([0, 1, 255, 256, 4097, M - 1])
    if variant == "forward":
        check("y", host(outs[0])[rows], oracle.linear_forward(x[rows], w, b), "bf16")
    else:
        check("dX", host(outs[0])[rows], oracle.linear_input_grad(gy[rows], w), "bf16")
