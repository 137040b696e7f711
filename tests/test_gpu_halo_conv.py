"""The halo convolution path: stride-1 convolutions of 64-channel inputs whose
filter fits in LDS (the 3x3 64 -> 64 layers of a ResNet stage 1, forward and
input gradient), stride-2 ones through their four stride phases (the stage's
downsampling layer: the forward over the input's phases, the input gradient
over its own) and a 3-channel stride-2 stem through its 2x2-block form: the
forward as a 4x4 stride-1 convolution of 16-channel blocks, the input gradient
as a 4x4 stride-1 correlation of the 64-channel dy.  Each
case runs with the halo kernel and with it switched off
(MEMSAVE_CONV_HALO=off, the implicit GEMM), both against the oracle, on
ragged tile grids, widths below and above one 32-wide column tile, zero
padding on every edge and every flag."""
import os

import pytest

import oracle
import paper_2404_12406_amd as ms
import synth

from _gpu import check, dev, host

pytestmark = pytest.mark.gpu

CASES = [
    # x shape, w shape, stride, pad
    ((2, 64, 13, 11), (64, 64, 3, 3), (1, 1), (1, 1)),     # ragged rows and columns
    ((1, 64, 9, 40), (64, 64, 3, 3), (1, 1), (1, 1)),      # two column tiles of 20
    ((3, 64, 7, 8), (64, 64, 3, 3), (1, 1), (1, 1)),       # narrow image
    ((1, 64, 56, 56), (64, 64, 3, 3), (1, 1), (1, 1)),     # the ResNet stage-1 tile shape
    ((2, 64, 10, 12), (32, 64, 3, 3), (1, 1), (0, 2)),     # 32 outputs: the 16-tap kernel; asymmetric pad
    ((2, 64, 11, 9), (24, 64, 2, 3), (1, 1), (1, 0)),      # 24 outputs (not a power of two), 2 x 3 taps
    ((2, 64, 10, 9), (48, 64, 2, 3), (1, 1), (1, 1)),      # 48 outputs, 2 x 3 taps: the generic 64-column loop
    ((2, 40, 9, 11), (64, 40, 2, 2), (1, 1), (1, 1)),      # input gradient of 40 channels, 2 x 2 taps
    ((1, 16, 12, 14), (64, 16, 4, 4), (1, 1), (0, 3)),     # input gradient only: 16 channels, 4 x 4 taps
    ((2, 3, 37, 41), (64, 3, 7, 7), (2, 2), (3, 3)),       # stem: both ways through 2 x 2 blocks
    ((2, 2, 21, 18), (48, 2, 7, 7), (2, 2), (3, 3)),       # 16-channel blocks: 48 outputs, 2 input channels
    ((2, 3, 30, 32), (64, 3, 7, 7), (2, 2), (3, 3)),       # stem with rows of 16-byte vectors: row-staged packing
    ((1, 4, 19, 20), (48, 4, 7, 7), (2, 2), (3, 3)),       # 4 channels, odd height, row-staged packing
    # stride 2, forward through the four stride phases
    ((2, 64, 23, 21), (64, 64, 3, 3), (2, 2), (1, 1)),     # odd input: 12 x 11 outputs, ragged tiles
    ((1, 64, 112, 112), (64, 64, 3, 3), (2, 2), (1, 1)),   # the ResNet stage-1 downsampling layer, one image
    ((2, 64, 16, 70), (40, 64, 3, 3), (2, 2), (0, 1)),     # 40 outputs, two column tiles, asymmetric pad
    ((2, 64, 14, 15), (64, 64, 2, 2), (2, 2), (0, 0)),     # 2 x 2 taps: one tap per phase, no padding
    ((1, 64, 20, 22), (32, 64, 3, 1), (2, 2), (1, 0)),     # 3 x 1 taps, 32 outputs
    # stride 2, input gradient through the four output phases (64 output-gradient channels)
    ((2, 40, 17, 19), (64, 40, 3, 3), (2, 2), (1, 1)),     # 40 input channels, odd extents
    ((1, 24, 17, 9), (64, 24, 3, 3), (2, 2), (2, 2)),      # padding 2: the halo starts one pixel early
    ((1, 32, 18, 18), (64, 32, 2, 3), (2, 2), (1, 1)),     # 2 x 3 taps: one and two taps per phase row
]


@pytest.fixture(params=["halo", "off"])
def halo(request):
    old = os.environ.get("MEMSAVE_CONV_HALO")
    if request.param == "off":
        os.environ["MEMSAVE_CONV_HALO"] = "off"
    yield request.param
    if old is None:
        os.environ.pop("MEMSAVE_CONV_HALO", None)
    else:
        os.environ["MEMSAVE_CONV_HALO"] = old


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("mask", [7, 1])
def test_halo_conv(case, mask, halo):
    xs, ws, stride, pad = CASES[case]
    seed = 8100 + 10 * case + mask
    x = synth.normal(xs, seed, dtype="bf16")
    w = synth.kaiming_uniform(ws, seed + 1, ws[1] * ws[2] * ws[3], dtype="bf16")
    b = synth.normal((ws[0],), seed + 2, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.Conv2d(stride, pad), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), mask)
    y_ref = oracle.conv2d_forward(x, w, b, stride, pad)
    assert oracle.rel_err(oracle.conv2d_forward(x, w, None, stride, pad), y_ref) > 0.2
    check("y", host(y), y_ref, "bf16")
    gy = synth.normal(tuple(y.shape), seed + 3, dtype="bf16")
    grads = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(grads[0]), oracle.conv2d_input_grad(gy, w, xs, stride, pad), "bf16")
    if mask == 7:
        check("dW", host(grads[1]), oracle.conv2d_weight_grad(gy, x, ws, stride, pad), "bf16")
        check("db", host(grads[2]), oracle.conv2d_bias_grad(gy), "bf16")


def test_halo_transposed_conv_forward():
    """A stride-1 transposed convolution's forward is the input gradient of
    the convolution it is the adjoint of: 64 input channels reach the halo
    kernel with the bias added in its epilogue."""
    xs, co = (2, 64, 9, 13), 64
    x = synth.normal(xs, 8190, dtype="bf16")
    w = synth.kaiming_uniform((64, co, 3, 3), 8191, co * 9, dtype="bf16")
    b = synth.normal((co,), 8192, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.ConvTranspose2d(1, 1), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    check("y", host(y), oracle.convt2d_forward(x, w, b, (1, 1), (1, 1), (0, 0)), "bf16")
    gy = synth.normal(tuple(y.shape), 8193, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(gx), oracle.convt2d_input_grad(gy, w, xs, (1, 1), (1, 1)), "bf16")
    check("dW", host(gw), oracle.convt2d_weight_grad(gy, x, (64, co, 3, 3), (1, 1), (1, 1)), "bf16")
    check("db", host(gb), oracle.convt2d_bias_grad(gy), "bf16")


def test_halo_transposed_conv_forward_stride_2():
    """A stride-2 transposed convolution of 64 input channels (3x3, pad 1,
    output padding 1: 2x upsampling) runs its forward through the output
    phases of the adjoint convolution's input gradient, bias in the
    epilogue."""
    xs, co = (2, 64, 9, 13), 48
    x = synth.normal(xs, 8194, dtype="bf16")
    w = synth.kaiming_uniform((64, co, 3, 3), 8195, co * 9, dtype="bf16")
    b = synth.normal((co,), 8196, 1.0, dtype="bf16")
    y, rec = ms.layer_forward(ms.ConvTranspose2d(2, 1, 1), dev(x, "bf16"), dev(w, "bf16"), dev(b, "bf16"), 7)
    assert tuple(y.shape) == (2, co, 18, 26)
    check("y", host(y), oracle.convt2d_forward(x, w, b, (2, 2), (1, 1), (1, 1)), "bf16")
    gy = synth.normal(tuple(y.shape), 8197, dtype="bf16")
    gx, gw, gb = ms.layer_backward(rec, dev(gy, "bf16"))
    check("dx", host(gx), oracle.convt2d_input_grad(gy, w, xs, (2, 2), (1, 1), (1, 1)), "bf16")
    check("dW", host(gw), oracle.convt2d_weight_grad(gy, x, (64, co, 3, 3), (2, 2), (1, 1), (1, 1)), "bf16")
    check("db", host(gb), oracle.convt2d_bias_grad(gy), "bf16")
