"""ReLU with a 1-bit saved mask (Sec. 2.2.2) on the GPU against the oracle:
y, the mask (every byte of the word-rounded buffer) and dx are bit-exact,
on ragged 1-D, 2-D and channels-last 4-D tensors, both dtypes, special
values, misaligned pointers (the scalar path), guard bands, mask 0, a
prepared layer reused, a Linear -> ReLU -> Linear chain whose ledger holds
only the mask, and sampled checks at the benchmark's size."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2404_12406_amd as ms
from paper_2404_12406_amd import _lib, api
import synth

from _gpu import TORCH_DT, dev, host

pytestmark = pytest.mark.gpu


def _special(n, dtype, seed):
    """N(0,1) draws (rounded to dtype) with zeros, -0, NaN, +-inf and
    subnormals of the dtype sprinkled in."""
    rng = np.random.default_rng(seed)
    x = synth.normal((n,), seed, dtype=dtype).astype(np.float64)
    sub = 1e-40 if dtype == "f32" else 2e-39   # subnormal in fp32 and in bf16
    vals = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, sub, -sub])
    k = min(n, max(1, n // 16))
    pos = rng.choice(n, size=k, replace=False)
    x[pos] = vals[rng.integers(0, vals.size, size=k)]
    return oracle.round_to(x, dtype) if dtype == "bf16" else x.astype(np.float32).astype(np.float64)


def _to_dev(a, dtype, shape):
    t = torch.from_numpy(np.ascontiguousarray(a.reshape(shape), dtype=np.float32)).to(TORCH_DT[dtype])
    if len(shape) == 4:
        t = t.contiguous(memory_format=torch.channels_last)
    return t.cuda()


def _same(got, want):
    """Bit-level equality of float64 views: NaN positions, values, and the
    sign of zeros."""
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    if not np.array_equal(np.isnan(got), np.isnan(want)):
        return False
    m = ~np.isnan(want)
    return np.array_equal(got[m], want[m]) and np.array_equal(np.signbit(got[m]), np.signbit(want[m]))


def _bits_bytes(bits: torch.Tensor) -> np.ndarray:
    return bits.cpu().numpy().view(np.uint8)


SHAPES = [(1,), (7,), (8,), (31,), (33,), (100003,), (37, 129), (2, 13, 9, 7), (3, 24, 17, 11)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_relu_forward_mask_backward_bit_exact(dtype, shape):
    n = int(np.prod(shape))
    seed = 9000 + n
    x = _special(n, dtype, seed).reshape(shape)
    xd = _to_dev(x, dtype, shape)
    y, rec = ms.layer_forward(ms.ReLU(), xd, mask=ms.MASK_INPUT)
    assert _same(host(y), oracle.relu_forward(x))
    layout = "nhwc" if len(shape) == 4 else "plain"
    bits = rec.saved["bits"]
    assert _bits_bytes(bits).tolist() == oracle.relu_mask_bits(oracle.memory_order(x, layout)).tolist()
    assert rec.account()["saved_activation_bytes"] == oracle.relu_mask_nbytes(n) == ms.relu_mask_bytes(n)
    gy = synth.normal(shape, seed + 1, dtype=dtype)
    (gx, gw, gb) = ms.layer_backward(rec, _to_dev(gy, dtype, shape))
    assert gw is None and gb is None
    assert _same(host(gx), oracle.relu_backward(gy, x))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [5, 64, 1000])
def test_relu_misaligned_pointers_take_the_scalar_path(dtype, n):
    x = _special(n, dtype, 9100 + n)
    buf = torch.zeros(n + 3, dtype=TORCH_DT[dtype], device="cuda")
    buf[1:n + 1] = torch.from_numpy(x.astype(np.float32)).to(TORCH_DT[dtype]).cuda()
    xv = buf[1:n + 1]                              # 2 or 4 bytes past a 16-byte boundary
    ybuf = torch.full((n + 3,), float("nan"), dtype=TORCH_DT[dtype], device="cuda")
    yv = ybuf[2:n + 2]
    y, rec = ms.layer_forward(ms.ReLU(), xv, mask=ms.MASK_INPUT, y=yv)
    assert _same(host(yv), oracle.relu_forward(x))
    assert torch.isnan(ybuf[:2]).all() and torch.isnan(ybuf[n + 2:]).all()
    assert _bits_bytes(rec.saved["bits"]).tolist() == oracle.relu_mask_bits(x).tolist()
    gy = synth.normal((n,), 9200 + n, dtype=dtype)
    gbuf = torch.zeros(n + 1, dtype=TORCH_DT[dtype], device="cuda")
    gbuf[1:] = torch.from_numpy(gy.astype(np.float32)).to(TORCH_DT[dtype]).cuda()
    dxbuf = torch.full((n + 2,), float("nan"), dtype=TORCH_DT[dtype], device="cuda")
    ms.layer_backward(rec, gbuf[1:], grad_x=dxbuf[1:n + 1])
    assert _same(host(dxbuf[1:n + 1]), oracle.relu_backward(gy, x))
    assert torch.isnan(dxbuf[0]) and torch.isnan(dxbuf[n + 1])


@pytest.mark.parametrize("n", [1, 33, 4097])
def test_relu_mask_buffer_guard_words_and_padding(n):
    """The library writes exactly ms_relu_mask_bytes(n) bytes: the mask and
    its zero padding up to the word; guard words around it stay intact."""
    x = _special(n, "bf16", 9300 + n)
    xd = dev(x, "bf16")
    words = ms.relu_mask_bytes(n) // 4
    guard = torch.full((words + 4,), -1, dtype=torch.int32, device="cuda")   # all bits set
    bits = guard[2:2 + words]
    y = torch.empty_like(xd)
    lib = _lib.load()
    h = api._relu_forward(lib, xd, y, bits, ms.MASK_INPUT)
    torch.cuda.synchronize()
    g = guard.cpu().numpy()
    assert (g[:2] == -1).all() and (g[2 + words:] == -1).all()
    assert _bits_bytes(bits).tolist() == oracle.relu_mask_bits(x).tolist()
    lib.ms_record_free(h)


def test_relu_mask_zero_writes_y_only_and_records_nothing():
    x = _special(1000, "f32", 9400)
    live0, _ = ms.ledger_read()
    y, rec = ms.layer_forward(ms.ReLU(), dev(x, "f32"), mask=0)
    assert rec is None
    assert _same(host(y), oracle.relu_forward(x))
    assert ms.ledger_read()[0] == live0


def test_relu_prepared_layer_reuses_its_mask_buffer():
    shape = (4, 32, 6, 5)
    x1 = _special(int(np.prod(shape)), "bf16", 9500).reshape(shape)
    x2 = -x1
    xd = _to_dev(x1, "bf16", shape)
    gy = synth.normal(shape, 9501, dtype="bf16")
    gx = torch.empty_like(xd)
    p = ms.PreparedLayer(ms.ReLU(), xd, mask=ms.MASK_INPUT, grad_y=_to_dev(gy, "bf16", shape), grad_x=gx)
    for xa in (x1, x2):
        xd.copy_(_to_dev(xa, "bf16", shape))
        p.forward()
        assert p.account()["saved_activation_bytes"] == ms.relu_mask_bytes(xd.numel())
        assert _bits_bytes(p.bits).tolist() == oracle.relu_mask_bits(oracle.memory_order(xa, "nhwc")).tolist()
        p.backward()
        assert _same(host(gx), oracle.relu_backward(gy, xa))


def test_linear_relu_linear_chain_keeps_only_the_mask():
    """Sec. 2.2.2: a ReLU between two frozen linears with the input requiring
    grad; neither linear keeps its input (weights frozen) and the ReLU keeps
    one bit per element instead of its output."""
    from paper_2404_12406_amd.stack import Chain, LayerCall
    M, D, H = 96, 64, 136
    x = synth.normal((M, D), 9600, dtype="bf16")
    W1 = synth.normal((H, D), 9601, 0.1, dtype="bf16")
    b1 = synth.normal((H,), 9602, 0.1, dtype="bf16")
    W2 = synth.normal((D, H), 9603, 0.1, dtype="bf16")
    gy = synth.normal((M, D), 9604, dtype="bf16")
    calls = [LayerCall(ms.Linear(), dev(W1, "bf16"), dev(b1, "bf16"), ms.MASK_INPUT),
             LayerCall(ms.ReLU(), None, None, ms.MASK_INPUT),
             LayerCall(ms.Linear(), dev(W2, "bf16"), None, ms.MASK_INPUT)]
    ch = Chain(calls, dev(x, "bf16"), dev(gy, "bf16"))
    ms.ledger_reset()
    live0, _ = ms.ledger_read()
    ch.forward()
    torch.cuda.synchronize()
    live, peak = ms.ledger_read()
    assert live - live0 == ms.relu_mask_bytes(M * H)
    ch.backward()
    # the ReLU on the GPU's own hidden tensors is exact ...
    h1, a1 = host(ch.acts[1]), host(ch.acts[2])
    g1, g0 = host(ch.grads[2][0]), host(ch.grads[1][0])
    assert _same(a1, oracle.relu_forward(h1))
    assert _same(g0, oracle.relu_backward(g1, h1))
    # ... and the whole chain matches the oracle composition within bf16 tolerance
    h1o = oracle.round_to(oracle.linear_forward(x, W1, b1), "bf16")
    g1o = oracle.round_to(oracle.linear_input_grad(gy, W2), "bf16")
    gxo = oracle.linear_input_grad(oracle.round_to(oracle.relu_backward(g1o, h1o), "bf16"), W1)
    assert oracle.rel_err(host(ch.grads[0][0]), gxo) <= 2e-2


def test_relu_sampled_at_benchmark_size():
    """The benchmark's tensor (64 x 64 x 112 x 112 bf16, channels-last): y,
    mask bytes and dx on 65536 sampled 8-element groups."""
    shape = (64, 64, 112, 112)
    n = int(np.prod(shape))
    g = torch.Generator(device="cuda").manual_seed(9700)
    xd = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    y, rec = ms.layer_forward(ms.ReLU(), xd, mask=ms.MASK_INPUT)
    bits_t = rec.saved["bits"]     # the record releases it at backward; keep a reference to read it
    gyd = torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16).contiguous(memory_format=torch.channels_last)
    gx, _, _ = ms.layer_backward(rec, gyd)
    torch.cuda.synchronize()
    xm = torch.as_strided(xd, (n,), (1,)).float().cpu().numpy().astype(np.float64)
    ym = torch.as_strided(y, (n,), (1,)).float().cpu().numpy().astype(np.float64)
    gym = torch.as_strided(gyd, (n,), (1,)).float().cpu().numpy().astype(np.float64)
    gxm = torch.as_strided(gx, (n,), (1,)).float().cpu().numpy().astype(np.float64)
    bb = _bits_bytes(bits_t)
    rng = np.random.default_rng(9701)
    groups = np.unique(np.concatenate([rng.integers(0, n // 8, 65536), [0, n // 8 - 1]]))
    for j in groups:
        sl = slice(8 * j, 8 * j + 8)
        assert _same(ym[sl], oracle.relu_forward(xm[sl]))
        assert int(bb[j]) == int(oracle.relu_mask_bits(xm[sl])[0])
        assert _same(gxm[sl], oracle.relu_backward(gym[sl], xm[sl]))
    assert rec.account()["saved_activation_bytes"] == ms.relu_mask_bytes(n) == n // 8
