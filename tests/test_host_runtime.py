"""Host-only tests of the runtime (validation, save rule, records, ledger,
launch plan) and of the C ABI's exports.  No GPU: the runtime is linked with
stub launchers (tests/native/host_stub.cpp) that launch nothing and check
that every pointer a kernel would dereference for the requested outputs is
present.  The save rule is compared bit-exactly with the oracle's closed
form; the exports with every declaration in include/*.h."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2404_12406_amd._lib as L
from oracle import policy as P
from synth import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
BUILD = os.path.join(NATIVE, "_build")
STUB_SO = os.path.join(BUILD, "libmemsave_hoststub.so")
DT = {"f32": L.MS_F32, "bf16": L.MS_BF16}
KIND = {"conv2d": L.MS_CONV2D, "linear": L.MS_LINEAR, "bn_eval": L.MS_BN_EVAL, "avgpool": L.MS_AVGPOOL,
        "conv_transpose2d": L.MS_CONV_TRANSPOSE2D}
FAKE = 0x7f0000000000  # a 256-byte aligned address nobody dereferences


def _build_stub():
    os.makedirs(BUILD, exist_ok=True)
    srcs = [os.path.join(ROOT, "paper_2404_12406_amd", "csrc", "memsave.cpp"), os.path.join(NATIVE, "host_stub.cpp")]
    tmp = STUB_SO + f".tmp{os.getpid()}"
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-Wall", "-I", os.path.join(ROOT, "include"),
                    *srcs, "-o", tmp], check=True)
    os.replace(tmp, STUB_SO)


@pytest.fixture(scope="module")
def stub():
    _build_stub()
    lib = L.configure(ctypes.CDLL(STUB_SO))
    lib.stub_log.restype = ctypes.c_char_p
    lib.stub_violations.restype = ctypes.c_char_p
    return lib


# ------------------------------------------------------------------ helpers
def tdesc(shape, dtype="bf16", layout="auto", data=True, addr=FAKE):
    t = L.MsTensor()
    t.data = addr if data else None
    t.dtype = DT[dtype] if isinstance(dtype, str) else dtype
    t.ndim = len(shape)
    for i, s in enumerate(shape):
        t.shape[i] = s
    if len(shape) == 4 and layout in ("auto", "nhwc"):
        N, C, H, W = shape
        st = (H * W * C, 1, W * C, C)
    elif len(shape) == 5 and layout in ("auto", "nhwc"):
        N, C, D, H, W = shape
        st = (D * H * W * C, 1, H * W * C, W * C, C)
    else:
        st, acc = [], 1
        for s in reversed(shape):
            st.append(acc)
            acc *= max(s, 1)
        st = tuple(reversed(st))
    for i, s in enumerate(st):
        t.stride[i] = s
    return t


def ref(t):
    return ctypes.byref(t) if t is not None else None


class LayerArgs:
    """MsLayer + tensors of one layer description (fake device pointers)."""

    def __init__(self, spec: wl.LayerSpec, dtype, data=True, addr=FAKE):
        self.spec = spec
        self.layer = L.MsLayer()
        self.layer.kind = KIND[spec.kind]
        self.layer.stride[0], self.layer.stride[1] = spec.stride
        self.layer.pad[0], self.layer.pad[1] = spec.pad
        self.layer.out_pad[0], self.layer.out_pad[1] = spec.out_pad
        self.layer.eps = spec.eps
        self.x = tdesc(spec.in_shape, dtype, data=data, addr=addr)
        ws = spec.weight_shape()
        self.W = tdesc(ws, dtype, data=data, addr=addr) if ws is not None else None
        has_b = spec.has_bias and spec.kind != "avgpool"
        self.b = tdesc((spec.out_ch if spec.kind != "bn_eval" else spec.in_shape[1],), dtype, data=data, addr=addr) if has_b else None
        self.y = tdesc(spec.out_shape(), dtype, data=data, addr=addr)
        if spec.kind == "bn_eval":
            C = spec.in_shape[1]
            self.mean = tdesc((C,), dtype, data=data, addr=addr)
            self.var = tdesc((C,), dtype, data=data, addr=addr)
            self.layer.running_mean = ctypes.pointer(self.mean)
            self.layer.running_var = ctypes.pointer(self.var)


def _numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


def _all_layers():
    out = []
    for name, w in wl.all_workloads().items():
        seen = set()
        for l in w.layers:
            key = (l.kind, l.in_shape, l.out_ch, l.ksize, l.stride, l.pad, l.has_bias)
            if key in seen:
                continue
            seen.add(key)
            out.append((f"{name}:{l.name}", l, w.dtype))
    return out


ALL_LAYERS = _all_layers()


# ------------------------------------------------------------------ exports
def _declared(headers):
    names = set()
    for h in headers:
        txt = open(h).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        names |= set(re.findall(r"\b(ms_[a-z_]+)\s*\(", txt))
    return names


def test_headers_declare_what_the_binding_knows():
    hdrs = [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h")]
    assert _declared(hdrs) == set(L.EXPORTS)


def test_library_exports_every_declared_symbol():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libmemsave.so not built")
    hdrs = [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h")]
    lib = ctypes.CDLL(L.LIB_PATH)
    for name in _declared(hdrs):
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True, text=True).stdout
    for name in _declared(hdrs):
        assert re.search(rf"\bT {name}$", out, re.M), name


def test_real_library_policy_without_gpu():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libmemsave.so not built")
    lib = L.load()
    spec = wl.single_conv_f32().layers[0]
    a = LayerArgs(spec, "f32", data=False)
    acct = L.MsAccount()
    assert lib.ms_policy_account(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), 1, 1, ctypes.byref(acct)) == 0
    assert acct.saved_activation_bytes == 524288
    assert lib.ms_version().decode().startswith("memsave")


# ------------------------------------------------------------------ save rule
@pytest.mark.parametrize("label,spec,dtype", ALL_LAYERS, ids=[a[0] for a in ALL_LAYERS])
def test_policy_account_matches_closed_form(stub, label, spec, dtype):
    a = LayerArgs(spec, dtype, data=False)
    masks = [0, 1] if spec.kind == "avgpool" else range(8)
    for mask in masks:
        if (mask & 4) and a.b is None:
            continue
        for pol in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE):
            acct = L.MsAccount()
            st = stub.ms_policy_account(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, pol,
                                        ctypes.byref(acct))
            assert st == 0, stub.ms_last_error()
            want = P.saved_activation_bytes(spec.kind, mask, _numel(spec.in_shape), dtype, pol,
                                            a.W is not None, a.b is not None)
            assert acct.saved_activation_bytes == want, (label, mask, pol)
            sv = P.saved_tensors(spec.kind, mask, pol, a.W is not None, a.b is not None)
            assert bool(acct.borrowed & L.MS_SAVED_X) == sv["x"]


# ------------------------------------------------------------------ records + plan
def _grads(a, mask):
    gx = tdesc(a.spec.in_shape, a.x.dtype) if mask & 1 else None
    gw = tdesc(a.spec.weight_shape(), a.x.dtype) if mask & 2 else None
    gb = tdesc((a.b.shape[0],), a.x.dtype) if mask & 4 else None
    return gx, gw, gb


@pytest.mark.parametrize("label,spec,dtype", ALL_LAYERS, ids=[a[0] for a in ALL_LAYERS])
def test_forward_backward_plan(stub, label, spec, dtype):
    a = LayerArgs(spec, dtype)
    masks = [0, 1] if spec.kind == "avgpool" else range(8)
    fwd_name = {"conv2d": "conv_fwd", "linear": "conv_fwd", "bn_eval": "bn_fwd", "avgpool": "avgpool_fwd",
                "conv_transpose2d": "conv_dgrad+bias" if spec.has_bias else "conv_dgrad"}[spec.kind]
    for mask in masks:
        if (mask & 4) and a.b is None:
            continue
        stub.stub_reset()
        live0, peak0 = ctypes.c_uint64(), ctypes.c_uint64()
        stub.ms_ledger_read(ctypes.byref(live0), ctypes.byref(peak0))
        h = ctypes.c_void_p()
        st = stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                   ctypes.byref(h), None)
        assert st == 0, stub.ms_last_error()
        assert stub.stub_log().decode() == fwd_name + ";"
        if mask == 0:
            assert not h.value
            continue
        acct = L.MsAccount()
        stub.ms_record_account(h, ctypes.byref(acct))
        want = P.saved_activation_bytes(spec.kind, mask, _numel(spec.in_shape), dtype, P.SELECTIVE)
        assert acct.saved_activation_bytes == want
        live, peak = ctypes.c_uint64(), ctypes.c_uint64()
        stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak))
        assert live.value - live0.value == want
        stub.stub_reset()
        gy = tdesc(spec.out_shape(), dtype)
        gx, gw, gb = _grads(a, mask)
        st = stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None)
        assert st == 0, (stub.ms_last_error(), stub.stub_violations())
        assert stub.stub_violations().decode() == ""
        log = stub.stub_log().decode().split(";")[:-1]
        plan = P.launched(spec.kind, mask)
        if spec.kind in ("conv2d", "linear"):
            assert ("conv_dgrad" in log) == plan["dgrad"]
            assert ("conv_wgrad" in log or "conv_wgrad+db" in log) == plan["wgrad"]
            # the bias gradient comes from a column sum, or fused into the
            # weight-gradient GEMM when that runs in bf16 -- never both
            fused = "conv_wgrad+db" in log
            assert (("colsum" in log) or fused) == plan["bgrad"]
            assert not (fused and "colsum" in log)
        elif spec.kind == "conv_transpose2d":
            assert log == [n for n, f in (("conv_fwd", "dgrad"), ("conv_wgrad", "wgrad"), ("colsum", "bgrad"))
                           if plan[f]]
        elif spec.kind == "bn_eval":
            assert log == ["bn_bwd"]
        else:
            assert log == ["avgpool_bwd"]
        stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak))
        assert live.value == live0.value
        assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == L.MS_E_CONSUMED
        stub.ms_record_free(h)
    assert stub.ms_testing_live_records() == 0


def test_backward_rejects_grad_sets_that_contradict_the_mask(stub):
    spec = wl.conv_sweep_bf16("11").layers[0]
    a = LayerArgs(spec, "bf16")
    for mask in range(1, 8):
        h = ctypes.c_void_p()
        assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                     ctypes.byref(h), None) == 0
        gy = tdesc(spec.out_shape())
        for given in range(8):
            if given == mask:
                continue
            stub.stub_reset()
            gx, gw, gb = _grads(a, given)
            assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == L.MS_E_MASK
            assert stub.stub_log().decode() == ""          # nothing launched
        acct = L.MsAccount()
        stub.ms_record_account(h, ctypes.byref(acct))
        gx, gw, gb = _grads(a, mask)
        # wrong grad shape / dtype / layout are caught too
        if gx is not None:
            bad = tdesc((1, 2, 3, 4))
            assert stub.ms_layer_backward(h, ref(gy), ref(bad), ref(gw), ref(gb), None) == L.MS_E_SHAPE
            badl = tdesc(spec.in_shape)
            badl.stride[2] = 0                             # rows of dx would share memory
            assert stub.ms_layer_backward(h, ref(gy), ref(badl), ref(gw), ref(gb), None) == L.MS_E_LAYOUT
            badd = tdesc(spec.in_shape, "f32")
            assert stub.ms_layer_backward(h, ref(gy), ref(badd), ref(gw), ref(gb), None) == L.MS_E_DTYPE
        assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == 0
        stub.ms_record_free(h)


def test_forward_validation_errors_launch_nothing(stub):
    spec = wl.conv_sweep_bf16("11").layers[0]
    live0, pk = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live0), ctypes.byref(pk))

    def fwd(a, mask, x=None, W="keep", b="keep", y=None):
        h = ctypes.c_void_p()
        stub.stub_reset()
        st = stub.ms_layer_forward(ctypes.byref(a.layer), ref(x or a.x), ref(a.W if W == "keep" else W),
                                   ref(a.b if b == "keep" else b), mask, ref(y or a.y), ctypes.byref(h), None)
        assert stub.stub_log().decode() == "" and not h.value
        return st

    a = LayerArgs(spec, "bf16")
    assert fwd(a, 8) == L.MS_E_MASK
    assert fwd(a, 2, W=None) == L.MS_E_MASK
    assert fwd(a, 4, b=None) == L.MS_E_MASK
    negx = tdesc(spec.in_shape)
    negx.stride[3] = -negx.stride[3]
    assert fwd(a, 1, x=negx) == L.MS_E_LAYOUT
    ovy = tdesc(spec.out_shape())
    ovy.stride[0] = 1                                  # images would overlap
    assert fwd(a, 1, y=ovy) == L.MS_E_LAYOUT
    assert fwd(a, 1, x=tdesc(spec.in_shape, "f32")) == L.MS_E_DTYPE
    assert fwd(a, 1, x=tdesc((32, 128, 28, 28))) == L.MS_E_SHAPE
    assert fwd(a, 1, y=tdesc((32, 256, 27, 28))) == L.MS_E_SHAPE
    assert fwd(a, 1, x=tdesc(spec.in_shape, data=False)) == L.MS_E_NULL
    assert fwd(a, 1, x=tdesc(spec.in_shape, 7)) == L.MS_E_DTYPE
    a.layer.stride[0] = 0
    assert fwd(a, 1) == L.MS_E_ARG
    a.layer.stride[0] = 1
    a.layer.pad[0] = -1
    assert fwd(a, 1) == L.MS_E_ARG
    a.layer.pad[0] = 1
    big = LayerArgs(wl.LayerSpec("linear", "big", (70000, 40000), out_ch=8, has_bias=False), "bf16")
    assert fwd(big, 1) == L.MS_E_UNSUPPORTED
    pool = LayerArgs(wl.LayerSpec("avgpool", "p", (2, 8, 4, 4)), "bf16")
    assert fwd(pool, 2, W=None, b=None) == L.MS_E_MASK
    bn = LayerArgs(wl.resnet18_shaped_bf16(batch=2, image=32).layers[1], "bf16")
    bn.layer.running_var = None
    assert fwd(bn, 1) == L.MS_E_NULL
    assert "running_var" in stub.ms_last_error().decode()
    live = ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(pk))
    assert live.value == live0.value


def _nchw(shape, dtype="bf16"):
    return tdesc(shape, dtype, layout="nchw")


def test_tensors_in_other_layouts_are_staged_around_the_kernels(stub):
    """NCHW (any strides) at the boundary: every 4-D tensor that is not
    channels-last, and every matrix that is not row-major, is copied into a
    dense stand-in before the kernels run and copied out after them; the
    record still borrows the caller's own x, so its bytes are unchanged, and
    the accounting counts the stand-ins as transient workspace."""
    spec = wl.conv_sweep_bf16("11").layers[0]
    a = LayerArgs(spec, "bf16")
    xn, wn, yn = _nchw(spec.in_shape), _nchw(spec.weight_shape()), _nchw(spec.out_shape())
    for mask in range(8):
        h = ctypes.c_void_p()
        stub.stub_reset()
        assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(xn), ref(wn), ref(a.b), mask, ref(yn),
                                     ctypes.byref(h), None) == 0, stub.ms_last_error()
        assert stub.stub_log().decode() == "copy4;copy4;conv_fwd;copy4;"
        if mask == 0:
            continue
        acct = L.MsAccount()
        stub.ms_record_account(h, ctypes.byref(acct))
        assert acct.saved_activation_bytes == P.saved_activation_bytes("conv2d", mask, _numel(spec.in_shape), "bf16")
        hc = ctypes.c_void_p()
        assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                     ctypes.byref(hc), None) == 0
        accc = L.MsAccount()
        stub.ms_record_account(hc, ctypes.byref(accc))
        e = 2
        stage = (_numel(spec.out_shape()) * e                                    # grad_y
                 + ((mask >> 1) & 1) * (_numel(spec.in_shape) * e)                # x for the weight gradient
                 + (mask & 1) * (_numel(spec.weight_shape()) * e)                 # W for the input gradient
                 + (mask & 1) * (_numel(spec.in_shape) * e)                       # grad_x
                 + ((mask >> 1) & 1) * (_numel(spec.weight_shape()) * e))         # grad_W
        assert acct.transient_workspace_bytes - accc.transient_workspace_bytes == stage, mask
        stub.ms_record_free(hc)
        gy = _nchw(spec.out_shape())
        gx = _nchw(spec.in_shape) if mask & 1 else None
        gw = _nchw(spec.weight_shape()) if mask & 2 else None
        gb = tdesc((spec.out_ch,)) if mask & 4 else None
        stub.stub_reset()
        assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == 0, stub.ms_last_error()
        assert stub.stub_violations().decode() == ""
        log = stub.stub_log().decode().split(";")[:-1]
        n_in = 1 + ((mask >> 1) & 1) + (mask & 1)          # grad_y, x, W
        n_out = (mask & 1) + ((mask >> 1) & 1)             # grad_x, grad_W
        assert log[:n_in] == ["copy4"] * n_in and log[len(log) - n_out:] == ["copy4"] * n_out, log
        assert "copy4" not in log[n_in:len(log) - n_out]
        stub.ms_record_free(h)
    # a transposed matrix (Linear input [M, K] stored as K x M), BN-eval in NCHW
    lin = LayerArgs(wl.linear_stack_bf16(m=256).layers[0], "bf16")
    xt = tdesc((256, 1024))
    xt.stride[0], xt.stride[1] = 1, 256
    h = ctypes.c_void_p()
    stub.stub_reset()
    assert stub.ms_layer_forward(ctypes.byref(lin.layer), ref(xt), ref(lin.W), ref(lin.b), 5, ref(lin.y),
                                 ctypes.byref(h), None) == 0
    assert stub.stub_log().decode() == "copy4;conv_fwd;"
    stub.ms_record_free(h)
    bn = LayerArgs(wl.resnet18_shaped_bf16(batch=2, image=32).layers[1], "bf16")
    xb = _nchw(bn.spec.in_shape)
    stub.stub_reset()
    yb = _nchw(bn.spec.in_shape)
    assert stub.ms_layer_forward(ctypes.byref(bn.layer), ref(xb), ref(bn.W), ref(bn.b), 3, ref(yb), ctypes.byref(h),
                                 None) == 0
    assert stub.stub_log().decode() == "bn_nchw;"          # plain NCHW: swept in place
    stub.stub_reset()
    gb = _nchw(bn.spec.in_shape)
    assert stub.ms_layer_backward(h, ref(gb), ref(_nchw(bn.spec.in_shape)), ref(tdesc((bn.spec.in_shape[1],))), None,
                                  None) == 0, stub.ms_last_error()
    assert stub.stub_log().decode() == "copy4;copy4;bn_bwd;copy4;"   # the reduction: grad_y, x (dgamma); grad_x out
    stub.ms_record_free(h)
    assert stub.ms_layer_forward(ctypes.byref(bn.layer), ref(xb), ref(bn.W), ref(bn.b), 1, ref(yb), ctypes.byref(h),
                                 None) == 0
    acct = L.MsAccount()
    stub.ms_record_account(h, ctypes.byref(acct))
    stub.stub_reset()
    assert stub.ms_layer_backward(h, ref(gb), ref(_nchw(bn.spec.in_shape)), None, None, None) == 0
    assert stub.stub_log().decode() == "bn_nchw_bwd;"      # dx alone: the same in-place sweep
    stub.ms_record_free(h)
    sl = _nchw(bn.spec.in_shape)
    sl.stride[0] *= 2                                       # a slice: staged
    stub.stub_reset()
    assert stub.ms_layer_forward(ctypes.byref(bn.layer), ref(sl), ref(bn.W), ref(bn.b), 0, ref(yb), ctypes.byref(h),
                                 None) == 0
    assert stub.stub_log().decode() == "copy4;bn_fwd;copy4;"
    # the 3-D kinds stay channels-last only
    assert stub.ms_testing_live_records() == 0


def test_elementwise_layers_take_any_dense_layout(stub):
    """ReLU and dropout work in memory order: any dense layout (NCHW too) is
    taken as is, with y (and the gradients) in x's layout."""
    shape = (2, 16, 5, 7)
    x, y = _nchw(shape), _nchw(shape)
    h = ctypes.c_void_p()
    stub.stub_reset()
    assert stub.ms_relu_forward(ref(x), ref(y), FAKE, 1, ctypes.byref(h), None) == 0, stub.ms_last_error()
    assert stub.stub_log().decode() == "relu_fwd+bits;"
    assert stub.ms_layer_backward(h, ref(_nchw(shape)), ref(tdesc(shape)), None, None, None) == L.MS_E_LAYOUT
    assert stub.ms_layer_backward(h, ref(_nchw(shape)), ref(_nchw(shape)), None, None, None) == 0
    stub.ms_record_free(h)
    assert stub.ms_relu_forward(ref(x), ref(tdesc(shape)), FAKE, 1, ctypes.byref(h), None) == L.MS_E_LAYOUT
    sl = _nchw(shape)
    sl.stride[0] *= 2                                  # every other image of a larger tensor: not dense
    assert stub.ms_dropout_forward(ref(sl), ref(sl), ctypes.c_float(0.5), 1, 0, 1, ctypes.byref(h), None) == L.MS_E_LAYOUT


def test_workspace_failure_leaves_record_and_ledger_intact(stub):
    spec = wl.conv_sweep_bf16("01").layers[0]          # W and B trainable: keeps x, needs workspace
    a = LayerArgs(spec, "bf16")
    h = ctypes.c_void_p()
    assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), 6, ref(a.y),
                                 ctypes.byref(h), None) == 0
    live1, pk = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live1), ctypes.byref(pk))
    gy = tdesc(spec.out_shape())
    _, gw, gb = _grads(a, 6)
    stub.ms_testing_fail_next_workspace(1)
    stub.stub_reset()
    assert stub.ms_layer_backward(h, ref(gy), None, ref(gw), ref(gb), None) == L.MS_E_NOMEM
    assert stub.stub_log().decode() == ""
    live2 = ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live2), ctypes.byref(pk))
    assert live2.value == live1.value
    assert stub.ms_layer_backward(h, ref(gy), None, ref(gw), ref(gb), None) == 0   # retry succeeds
    stub.ms_record_free(h)
    stub.ms_record_free(None)


def test_noalloc_backward_launches_the_same_plan_from_the_fixed_scratch(stub):
    """The no-allocation backward runs the launch plan of ms_layer_backward
    with its workspace taken from the fixed scratch (never the allocating
    pool), rejects a workspace larger than the scratch before launching
    anything, and leaves that record usable by ms_layer_backward."""
    stub.stub_workspace_allocations.restype = ctypes.c_long
    cap = stub.ms_noalloc_scratch_bytes()
    assert cap == 64 << 20
    for spec, mask in ((wl.conv_sweep_bf16("01").layers[0], 6), (wl.linear_stack_bf16().layers[0], 5),
                       (wl.conv_sweep_bf16("11", pointwise=True).layers[0], 7)):
        a = LayerArgs(spec, "bf16")
        logs = []
        for entry in (stub.ms_layer_backward, stub.ms_layer_backward_noalloc):
            h = ctypes.c_void_p()
            assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                         ctypes.byref(h), None) == 0
            gy = tdesc(spec.out_shape())
            gx, gw, gb = _grads(a, mask)
            n_alloc = stub.stub_workspace_allocations()
            stub.stub_reset()
            assert entry(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == 0, stub.ms_last_error()
            assert stub.stub_violations().decode() == ""
            logs.append(stub.stub_log().decode())
            if entry is stub.ms_layer_backward_noalloc:
                assert stub.stub_workspace_allocations() == n_alloc
            stub.ms_record_free(h)
        acct_ws = logs[1].startswith("scratch;")
        assert logs[1] == ("scratch;" if acct_ws else "") + logs[0], logs
    # a backward whose workspace exceeds the scratch: the weight gradient of
    # a 4096 x 4096 Linear over 8192 rows (split-K partials)
    big = wl.LayerSpec("linear", "big", (8192, 4096), out_ch=4096, has_bias=True)
    a = LayerArgs(big, "bf16")
    h = ctypes.c_void_p()
    assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), 6, ref(a.y),
                                 ctypes.byref(h), None) == 0
    acct = L.MsAccount()
    stub.ms_record_account(h, ctypes.byref(acct))
    assert acct.transient_workspace_bytes > cap
    live1, pk = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live1), ctypes.byref(pk))
    gy = tdesc(big.out_shape())
    _, gw, gb = _grads(a, 6)
    stub.stub_reset()
    assert stub.ms_layer_backward_noalloc(h, ref(gy), None, ref(gw), ref(gb), None) == L.MS_E_UNSUPPORTED
    assert "scratch" in stub.ms_last_error().decode()
    assert stub.stub_log().decode() == ""
    live2 = ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live2), ctypes.byref(pk))
    assert live2.value == live1.value
    assert stub.ms_layer_backward(h, ref(gy), None, ref(gw), ref(gb), None) == 0
    stub.ms_record_free(h)


def test_ledger_peak_over_a_stack(stub):
    """Peak retained bytes of the ResNet-18-shaped stack in its 'Input'
    variant equal the closed form: convs and BN keep nothing, the final
    Linear keeps its input."""
    w = wl.resnet18_shaped_bf16(input_requires_grad=True)
    stub.ms_ledger_reset()
    live0, pk = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live0), ctypes.byref(pk))
    stub.ms_ledger_reset()
    hs = []
    for spec in w.layers:
        a = LayerArgs(spec, "bf16")
        h = ctypes.c_void_p()
        assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), spec.mask, ref(a.y),
                                     ctypes.byref(h), None) == 0
        hs.append(h)
    live, peak = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak))
    layers = [(l.kind, l.mask, _numel(l.in_shape), "bf16", l.kind != "avgpool", l.has_bias) for l in w.layers]
    assert peak.value - live0.value == P.stack_saved_bytes(layers, P.SELECTIVE) == 65536
    for h in hs:
        stub.ms_record_free(h)
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak))
    assert live.value == live0.value


def test_fast_path_operand_limit():
    """The bf16 GEMM fast path takes an operand only while its byte size stays
    below the out-of-range offset its loads use (and its row bases fit 32
    bits); larger operands -- e.g. the 8-channel padded copy of a 3-channel
    image of 2^28 pixels -- go to the general kernel."""
    src = os.path.join(BUILD, "limits_check.cpp")
    exe = os.path.join(BUILD, "limits_check")
    os.makedirs(BUILD, exist_ok=True)
    with open(src, "w") as f:
        f.write('#include "kernels/limits.h"\n#include <cstdio>\nusing namespace ms::g2;\n'
                "int main() {\n"
                "  const long long v[] = {0, 1, 2147483632LL, 2147483633LL, 2147483647LL, (1LL << 28) * 8, 64LL * 224 * 115 * 8, -1};\n"
                '  for (long long e : v) printf("%lld %d\\n", e, (int)operand_fits(e));\n'
                "  return 0;\n}\n")
    subprocess.run(["g++", "-std=c++17", "-I", os.path.join(ROOT, "paper_2404_12406_amd", "csrc"), src, "-o", exe],
                   check=True)
    out = dict(tuple(map(int, l.split())) for l in subprocess.run([exe], capture_output=True, text=True,
                                                                   check=True).stdout.split("\n") if l)
    # the largest operand whose last byte stays below 0xFFFFFFF0 with 8 elements of slack
    assert out[2147483632] == 1 and out[2147483633] == 0
    assert out[2147483647] == 0 and out[(1 << 28) * 8] == 0 and out[-1] == 0
    assert out[0] == 1 and out[64 * 224 * 115 * 8] == 1       # the stem's packed input
    assert 2147483632 * 2 + 16 <= 0xFFFFFFF0


def test_native_driver_under_sanitizers():
    """The same lifecycle driven from C++ with AddressSanitizer and UBSan."""
    exe = os.path.join(BUILD, "test_host_runtime")
    os.makedirs(BUILD, exist_ok=True)
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "paper_2404_12406_amd", "csrc", "memsave.cpp"),
                    os.path.join(NATIVE, "host_stub.cpp"), os.path.join(NATIVE, "test_host_runtime.cpp"), "-o", exe],
                   check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ALL OK" in r.stdout


EDGE_SPECS = [
    wl.LayerSpec("linear", "k0", (5, 0), out_ch=6, has_bias=True),
    wl.LayerSpec("linear", "odd", (129, 30), out_ch=20, has_bias=True),
    wl.LayerSpec("linear", "one", (1, 1), out_ch=1, has_bias=True),
    wl.LayerSpec("linear", "m0", (0, 16), out_ch=8, has_bias=True),
    wl.LayerSpec("conv2d", "n0", (0, 16, 8, 8), out_ch=8, ksize=(3, 3), pad=(1, 1), has_bias=True),
    wl.LayerSpec("conv2d", "c3", (2, 3, 30, 29), out_ch=16, ksize=(7, 7), stride=(2, 2), pad=(3, 3), has_bias=True),
    wl.LayerSpec("conv2d", "c12", (1, 12, 11, 13), out_ch=20, ksize=(3, 2), stride=(3, 2), pad=(0, 1), has_bias=True),
    wl.LayerSpec("conv2d", "big", (64, 512, 7, 7), out_ch=512, ksize=(3, 3), pad=(1, 1), has_bias=True),
    wl.LayerSpec("bn_eval", "bn13", (2, 13, 5, 6), has_bias=True),
    wl.LayerSpec("bn_eval", "bn0", (0, 24, 5, 6), has_bias=True),
    wl.LayerSpec("bn_eval", "bn2d", (50, 36), has_bias=True),
]


@pytest.mark.parametrize("spec", EDGE_SPECS + [l for _, l, _ in ALL_LAYERS], ids=lambda s: s.name)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_real_library_planners_on_edge_shapes(spec, dtype):
    """ms_policy_account runs the real launch planners (split-K and
    reduction workspace sizing) without touching the GPU: every mask and
    policy must return a result on degenerate and ragged shapes."""
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libmemsave.so not built")
    lib = L.load()
    a = LayerArgs(spec, dtype, data=False)
    for mask in ([0, 1] if spec.kind == "avgpool" else range(8)):
        if (mask & 4) and a.b is None:
            continue
        for pol in (0, 1, 2):
            acct = L.MsAccount()
            st = lib.ms_policy_account(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, pol,
                                       ctypes.byref(acct))
            assert st == 0, lib.ms_last_error()
            if mask & 4 and pol == 0:          # bias / beta gradients reduce through partials
                assert acct.transient_workspace_bytes > 0


def test_profile_api_validates_arguments(stub):
    n, t = ctypes.c_uint64(), ctypes.c_double()
    stub.ms_profile_start.argtypes = [ctypes.c_uint32]
    assert stub.ms_profile_start(64) == L.MS_E_ARG
    assert stub.ms_profile_start(L.MS_PROF_RED) == 0
    assert stub.ms_profile_read(L.MS_PROF_RED, ctypes.byref(n), ctypes.byref(t)) == 0
    assert stub.ms_profile_start(L.MS_PROF_FWD | L.MS_PROF_DGRAD) == 0
    assert stub.ms_profile_read(L.MS_PROF_FWD | L.MS_PROF_DGRAD, ctypes.byref(n), ctypes.byref(t)) == L.MS_E_ARG
    assert stub.ms_profile_read(L.MS_PROF_FWD, None, ctypes.byref(t)) == L.MS_E_NULL
    assert stub.ms_profile_read(L.MS_PROF_BN, ctypes.byref(n), ctypes.byref(t)) == 0
    assert stub.ms_profile_start(0) == 0


# ------------------------------------------------------------------ ReLU (Sec. 2.2.2)
def _relu_forward(stub, x, y, bits, mask):
    h = ctypes.c_void_p()
    st = stub.ms_relu_forward(ref(x), ref(y), ctypes.c_void_p(bits) if bits is not None else None, mask,
                              ctypes.byref(h), None)
    return st, h


@pytest.mark.parametrize("shape", [(1000,), (1,), (33, 7), (2, 16, 5, 7), (64, 64, 112, 112), (0,), (4, 0)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relu_record_keeps_one_bit_per_element(stub, shape, dtype):
    n = _numel(shape)
    x, y = tdesc(shape, dtype), tdesc(shape, dtype)
    stub.stub_reset()
    live0, peak0 = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live0), ctypes.byref(peak0))
    st, h = _relu_forward(stub, x, y, FAKE + 4096, L.MS_RG_INPUT)
    assert st == 0, stub.ms_last_error()
    assert stub.stub_violations().decode() == ""
    assert stub.ms_relu_mask_bytes(n) == P.relu_mask_bytes(n) == (4 * ((n + 31) // 32) if n else 0)
    acct = L.MsAccount()
    stub.ms_record_account(h, ctypes.byref(acct))
    assert acct.saved_activation_bytes == P.saved_activation_bytes("relu", 1, n, dtype, P.SELECTIVE)
    assert acct.borrowed == L.MS_SAVED_BITS and acct.kernels == L.MS_K_DGRAD
    assert acct.referenced_param_bytes == 0
    live = ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak0))
    assert live.value - live0.value == acct.saved_activation_bytes
    stub.stub_reset()
    gy, gx = tdesc(shape, dtype), tdesc(shape, dtype)
    assert stub.ms_layer_backward(h, ref(gy), ref(gx), None, None, None) == 0, stub.ms_last_error()
    assert stub.stub_log().decode() == "relu_bwd;"
    assert stub.stub_violations().decode() == ""
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(peak0))
    assert live.value == live0.value
    assert stub.ms_layer_backward(h, ref(gy), ref(gx), None, None, None) == L.MS_E_CONSUMED
    stub.ms_record_free(h)
    # mask 0: y only, no mask buffer needed, no record
    stub.stub_reset()
    st, h = _relu_forward(stub, x, y, None, 0)
    assert st == 0 and not h.value
    assert stub.stub_log().decode() in ("relu_fwd;", "")
    assert stub.ms_testing_live_records() == 0


def _sliced(shape):
    t = tdesc(shape, "bf16", "nchw")
    t.stride[0] *= 2
    return t


def test_relu_validation_errors_launch_nothing(stub):
    x, y = tdesc((8, 16), "bf16"), tdesc((8, 16), "bf16")
    cases = [
        (x, y, FAKE, L.MS_RG_WEIGHT, L.MS_E_MASK),
        (x, y, FAKE, L.MS_RG_INPUT | L.MS_RG_BIAS, L.MS_E_MASK),
        (x, y, None, L.MS_RG_INPUT, L.MS_E_NULL),
        (x, y, FAKE + 2, L.MS_RG_INPUT, L.MS_E_ARG),
        (x, tdesc((8, 17), "bf16"), FAKE, L.MS_RG_INPUT, L.MS_E_SHAPE),
        (x, tdesc((8, 16), "f32"), FAKE, L.MS_RG_INPUT, L.MS_E_DTYPE),
        (tdesc((2, 3, 4), "bf16"), tdesc((2, 3, 4), "bf16"), FAKE, L.MS_RG_INPUT, L.MS_E_SHAPE),
        (_sliced((2, 3, 4, 5)), _sliced((2, 3, 4, 5)), FAKE, 1, L.MS_E_LAYOUT),   # not dense
        (tdesc((2, 3, 4, 5), "bf16"), tdesc((2, 3, 4, 5), "bf16", "nchw"), FAKE, 1, L.MS_E_LAYOUT),
        (None, y, FAKE, L.MS_RG_INPUT, L.MS_E_NULL),
        (x, None, FAKE, L.MS_RG_INPUT, L.MS_E_NULL),
    ]
    for xi, yi, bits, mask, want in cases:
        stub.stub_reset()
        st, h = _relu_forward(stub, xi, yi, bits, mask)
        assert st == want, (mask, want, st, stub.ms_last_error())
        assert not h.value and stub.stub_log().decode() == ""
    # the generic entry point refuses ReLU (it has no slot for the mask buffer)
    layer = L.MsLayer()
    layer.kind = L.MS_RELU
    h = ctypes.c_void_p()
    assert stub.ms_layer_forward(ctypes.byref(layer), ref(x), None, None, 1, ref(y), ctypes.byref(h), None) == L.MS_E_ARG
    assert stub.ms_testing_live_records() == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relu_policy_account(stub, dtype):
    shape = (64, 64, 56, 56)
    n = _numel(shape)
    layer = L.MsLayer()
    layer.kind = L.MS_RELU
    x = tdesc(shape, dtype, data=False)
    for policy in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE):
        for mask in (0, 1):
            a = L.MsAccount()
            assert stub.ms_policy_account(ctypes.byref(layer), ref(x), None, None, mask, policy, ctypes.byref(a)) == 0
            assert a.saved_activation_bytes == P.saved_activation_bytes("relu", mask, n, dtype, policy)
    a = L.MsAccount()
    assert stub.ms_policy_account(ctypes.byref(layer), ref(x), ref(tdesc((4,), dtype)), None, 1, 0,
                                  ctypes.byref(a)) == L.MS_E_ARG


# ------------------------------------------------------------------ transposed convolution
class ConvTArgs:
    """MsLayer + tensors of a transposed convolution x[N,Ci,H,W], W[Ci,Co,R,S]."""

    def __init__(self, x_shape, Co, k, stride, pad, out_pad, dtype="bf16", bias=True, data=True):
        N, Ci, H, W = x_shape
        self.layer = L.MsLayer()
        self.layer.kind = L.MS_CONV_TRANSPOSE2D
        self.layer.stride[0], self.layer.stride[1] = stride
        self.layer.pad[0], self.layer.pad[1] = pad
        self.layer.out_pad[0], self.layer.out_pad[1] = out_pad
        Ho = (H - 1) * stride[0] - 2 * pad[0] + k[0] + out_pad[0]
        Wo = (W - 1) * stride[1] - 2 * pad[1] + k[1] + out_pad[1]
        self.x_shape, self.w_shape, self.y_shape = x_shape, (Ci, Co, k[0], k[1]), (N, Co, Ho, Wo)
        self.x = tdesc(x_shape, dtype, data=data)
        self.W = tdesc(self.w_shape, dtype, data=data)
        self.b = tdesc((Co,), dtype, data=data) if bias else None
        self.y = tdesc(self.y_shape, dtype, data=data)
        self.dtype = dtype


CONVT = [
    ((2, 16, 5, 7), 8, (4, 4), (2, 2), (1, 1), (0, 0)),
    ((1, 12, 6, 6), 3, (3, 3), (2, 2), (1, 1), (1, 1)),
    ((3, 8, 4, 5), 24, (2, 2), (2, 2), (0, 0), (0, 0)),
    ((1, 8, 1, 40), 8, (1, 3), (1, 1), (0, 1), (0, 0)),     # a 1-D transposed convolution
]


@pytest.mark.parametrize("case", range(len(CONVT)))
def test_conv_transpose_policy_matches_closed_form(stub, case):
    a = ConvTArgs(*CONVT[case], data=False)
    numel = _numel(a.x_shape)
    for mask in range(8):
        for pol in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE):
            acct = L.MsAccount()
            st = stub.ms_policy_account(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, pol,
                                        ctypes.byref(acct))
            assert st == 0, stub.ms_last_error()
            assert acct.saved_activation_bytes == P.saved_activation_bytes("conv_transpose2d", mask, numel,
                                                                           a.dtype, pol)
            sv = P.saved_tensors("conv_transpose2d", mask, pol)
            assert bool(acct.borrowed & L.MS_SAVED_X) == sv["x"]
            assert bool(acct.borrowed & L.MS_SAVED_W) == sv["W"]


@pytest.mark.parametrize("case", range(len(CONVT)))
def test_conv_transpose_forward_backward_plan(stub, case):
    """Forward: the input-gradient contraction (with the bias when there is
    one).  Backward: the forward contraction for dx, the weight-gradient
    contraction for dW (never with a fused bias: its column sums would be
    those of x), a column sum of grad_y for db -- each only under its flag."""
    for bias in (True, False):
        a = ConvTArgs(*CONVT[case], bias=bias)
        for mask in range(8):
            if (mask & 4) and not bias:
                continue
            stub.stub_reset()
            h = ctypes.c_void_p()
            st = stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                       ctypes.byref(h), None)
            assert st == 0, stub.ms_last_error()
            assert stub.stub_log().decode() == ("conv_dgrad+bias;" if bias else "conv_dgrad;")
            assert stub.stub_violations().decode() == ""
            if mask == 0:
                assert not h.value
                continue
            stub.stub_reset()
            gy = tdesc(a.y_shape)
            gx = tdesc(a.x_shape) if mask & 1 else None
            gw = tdesc(a.w_shape) if mask & 2 else None
            gb = tdesc((a.w_shape[1],)) if mask & 4 else None
            assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == 0, stub.ms_last_error()
            assert stub.stub_violations().decode() == ""
            want = [n for n, f in (("conv_fwd", 1), ("conv_wgrad", 2), ("colsum", 4)) if mask & f]
            assert stub.stub_log().decode().split(";")[:-1] == want
            stub.ms_record_free(h)
    assert stub.ms_testing_live_records() == 0


def test_conv_transpose_validation(stub):
    def fwd(a, mask=7, x=None, W=None, b="keep", y=None):
        h = ctypes.c_void_p()
        stub.stub_reset()
        st = stub.ms_layer_forward(ctypes.byref(a.layer), ref(x or a.x), ref(W or a.W),
                                   ref(a.b if b == "keep" else b), mask, ref(y or a.y), ctypes.byref(h), None)
        assert stub.stub_log().decode() == "" and not h.value
        return st

    a = ConvTArgs((2, 16, 5, 7), 8, (4, 4), (2, 2), (1, 1), (1, 0))
    assert fwd(a, y=tdesc((2, 8, 10, 14))) == L.MS_E_SHAPE        # out_pad ignored in y
    assert fwd(a, W=tdesc((8, 16, 4, 4))) == L.MS_E_SHAPE          # W given as [Co, Ci, R, S]
    negw = tdesc(a.w_shape)
    negw.stride[2] = -negw.stride[2]
    assert fwd(a, W=negw) == L.MS_E_LAYOUT          # other layouts are staged; negative strides are refused
    ovx = tdesc(a.y_shape)
    ovx.stride[0] = 0
    assert fwd(a, y=ovx) == L.MS_E_LAYOUT
    assert fwd(a, b=tdesc((16,))) == L.MS_E_SHAPE                  # bias has C_out entries
    assert fwd(a, x=tdesc(a.x_shape, "f32")) == L.MS_E_DTYPE
    a.layer.out_pad[0] = 2                                          # out_pad >= stride
    assert fwd(a) == L.MS_E_ARG
    a.layer.out_pad[0] = -1
    assert fwd(a) == L.MS_E_ARG
    a.layer.out_pad[0] = 1
    a.layer.stride[1] = 0
    assert fwd(a) == L.MS_E_ARG
    a.layer.stride[1] = 2
    # an output that would be empty: H = 1, R = 1, pad 1
    e = ConvTArgs((1, 8, 1, 4), 8, (1, 3), (1, 1), (0, 0), (0, 0))
    e.layer.pad[0] = 1
    assert fwd(e, y=tdesc((1, 8, 1, 6))) == L.MS_E_SHAPE
    # the forward is valid once everything matches
    h = ctypes.c_void_p()
    assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), 7, ref(a.y),
                                 ctypes.byref(h), None) == 0, stub.ms_last_error()
    stub.ms_record_free(h)


# ------------------------------------------------------------------ dropout
def _dropout_forward(lib, x, y, p, mask, seed=5, offset=0):
    h = ctypes.c_void_p()
    st = lib.ms_dropout_forward(ref(x), ref(y), p, seed, offset, mask, ctypes.byref(h), None)
    return st, h


@pytest.mark.parametrize("shape", [(1000,), (8, 16), (2, 3, 4, 5), (0, 7)])
@pytest.mark.parametrize("p", [0.0, 0.3, 1.0])
def test_dropout_record_keeps_no_device_memory(stub, shape, p):
    """Sec. 2.2.2: the record holds the generator state; backward launches
    the same pass on grad_y (all-zero output when p = 1)."""
    x, y = tdesc(shape, "bf16"), tdesc(shape, "bf16")
    live0, pk = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live0), ctypes.byref(pk))
    stub.stub_reset()
    st, h = _dropout_forward(stub, x, y, p, L.MS_RG_INPUT)
    assert st == 0, stub.ms_last_error()
    name = "dropout(all)" if p == 1.0 else "dropout"
    assert stub.stub_log().decode() == name + ";" and stub.stub_violations().decode() == ""
    a = L.MsAccount()
    stub.ms_record_account(h, ctypes.byref(a))
    assert a.saved_activation_bytes == 0 and a.borrowed == 0 and a.kernels == L.MS_K_DGRAD
    live, _ = ctypes.c_uint64(), ctypes.c_uint64()
    stub.ms_ledger_read(ctypes.byref(live), ctypes.byref(pk))
    assert live.value == live0.value
    stub.stub_reset()
    gy, gx = tdesc(shape, "bf16"), tdesc(shape, "bf16")
    assert stub.ms_layer_backward(h, ref(gy), ref(gx), None, None, None) == 0
    assert stub.stub_log().decode() == name + ";"
    stub.ms_record_free(h)
    # mask 0: the forward only, no record
    stub.stub_reset()
    st, h = _dropout_forward(stub, x, y, p, 0)
    assert st == 0 and not h.value
    assert stub.stub_log().decode() == name + ";"
    assert stub.ms_testing_live_records() == 0


def test_dropout_validation_errors_launch_nothing(stub):
    x, y = tdesc((8, 16), "bf16"), tdesc((8, 16), "bf16")
    cases = [
        (x, y, 0.5, L.MS_RG_WEIGHT, L.MS_E_MASK),
        (x, y, -0.1, 1, L.MS_E_ARG),
        (x, y, 1.5, 1, L.MS_E_ARG),
        (x, y, float("nan"), 1, L.MS_E_ARG),
        (x, y, float("inf"), 1, L.MS_E_ARG),
        (x, tdesc((8, 17), "bf16"), 0.5, 1, L.MS_E_SHAPE),
        (x, tdesc((8, 16), "f32"), 0.5, 1, L.MS_E_DTYPE),
        (_sliced((2, 3, 4, 5)), _sliced((2, 3, 4, 5)), 0.5, 1, L.MS_E_LAYOUT),
        (None, y, 0.5, 1, L.MS_E_NULL),
        (x, None, 0.5, 1, L.MS_E_NULL),
    ]
    for xi, yi, p, mask, want in cases:
        stub.stub_reset()
        st, h = _dropout_forward(stub, xi, yi, p, mask)
        assert st == want, (p, mask, want, st, stub.ms_last_error())
        assert not h.value and stub.stub_log().decode() == ""
    layer = L.MsLayer()
    layer.kind = L.MS_DROPOUT
    h = ctypes.c_void_p()
    assert stub.ms_layer_forward(ctypes.byref(layer), ref(x), None, None, 1, ref(y), ctypes.byref(h), None) == L.MS_E_ARG
    assert stub.ms_dropout_blocks(0) == 0 and stub.ms_dropout_blocks(4) == 1 and stub.ms_dropout_blocks(9) == 3
    assert stub.ms_testing_live_records() == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dropout_policy_account(stub, dtype):
    shape = (8192, 3072)
    n = _numel(shape)
    layer = L.MsLayer()
    layer.kind = L.MS_DROPOUT
    x = tdesc(shape, dtype, data=False)
    for policy in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE):
        for mask in (0, 1):
            a = L.MsAccount()
            assert stub.ms_policy_account(ctypes.byref(layer), ref(x), None, None, mask, policy, ctypes.byref(a)) == 0
            assert a.saved_activation_bytes == P.saved_activation_bytes("dropout", mask, n, dtype, policy)
            assert bool(a.borrowed & L.MS_SAVED_MASK8) == (policy == P.PYTORCH_DEFAULT and mask == 1)


# ------------------------------------------------------------------ 3-D convolutions
class Conv3dArgs:
    def __init__(self, x_shape, c_out, k, stride, pad, out_pad=None, dtype="bf16", bias=True, data=True):
        tr = out_pad is not None
        N, C, D, H, W = x_shape
        self.layer = L.MsLayer()
        self.layer.kind = L.MS_CONV_TRANSPOSE3D if tr else L.MS_CONV3D
        self.layer.stride_d, self.layer.stride[0], self.layer.stride[1] = stride
        self.layer.pad_d, self.layer.pad[0], self.layer.pad[1] = pad
        if tr:
            self.layer.out_pad_d, self.layer.out_pad[0], self.layer.out_pad[1] = out_pad
            out = [(e - 1) * s - 2 * p + kk + o for e, kk, s, p, o in zip((D, H, W), k, stride, pad, out_pad)]
            self.w_shape = (C, c_out) + tuple(k)
        else:
            out = [(e + 2 * p - kk) // s + 1 for e, kk, s, p in zip((D, H, W), k, stride, pad)]
            self.w_shape = (c_out, C) + tuple(k)
        self.x_shape, self.y_shape = x_shape, (N, c_out) + tuple(out)
        self.x = tdesc(x_shape, dtype, data=data)
        self.W = tdesc(self.w_shape, dtype, data=data)
        self.b = tdesc((c_out,), dtype, data=data) if bias else None
        self.y = tdesc(self.y_shape, dtype, data=data)
        self.dtype, self.tr = dtype, tr


CONV3D = [
    ((2, 8, 6, 7, 5), 16, (3, 3, 3), (1, 1, 1), (1, 1, 1), None),
    ((1, 3, 5, 8, 8), 8, (3, 1, 2), (2, 1, 2), (1, 0, 1), None),
    ((2, 16, 3, 4, 4), 8, (2, 4, 4), (2, 2, 2), (0, 1, 1), (1, 0, 1)),
    ((1, 8, 4, 5, 3), 3, (3, 3, 3), (1, 2, 1), (1, 1, 1), (0, 1, 0)),
]


@pytest.mark.parametrize("case", range(len(CONV3D)))
def test_conv3d_policy_and_plan(stub, case):
    a = Conv3dArgs(*CONV3D[case])
    kind = "conv_transpose3d" if a.tr else "conv3d"
    numel = _numel(a.x_shape)
    for mask in range(8):
        for pol in (P.SELECTIVE, P.PYTORCH_DEFAULT, P.ALL_TRUE):
            acct = L.MsAccount()
            assert stub.ms_policy_account(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, pol,
                                          ctypes.byref(acct)) == 0, stub.ms_last_error()
            assert acct.saved_activation_bytes == P.saved_activation_bytes(kind, mask, numel, a.dtype, pol)
        stub.stub_reset()
        h = ctypes.c_void_p()
        assert stub.ms_layer_forward(ctypes.byref(a.layer), ref(a.x), ref(a.W), ref(a.b), mask, ref(a.y),
                                     ctypes.byref(h), None) == 0, stub.ms_last_error()
        assert stub.stub_log().decode() == ("conv3d_dgrad+bias;" if a.tr else "conv3d_fwd;")
        if mask == 0:
            assert not h.value
            continue
        stub.stub_reset()
        gy = tdesc(a.y_shape)
        gx = tdesc(a.x_shape) if mask & 1 else None
        gw = tdesc(a.w_shape) if mask & 2 else None
        gb = tdesc((a.y_shape[1],)) if mask & 4 else None
        assert stub.ms_layer_backward(h, ref(gy), ref(gx), ref(gw), ref(gb), None) == 0, stub.ms_last_error()
        assert stub.stub_violations().decode() == ""
        log = stub.stub_log().decode().split(";")[:-1]
        if a.tr:
            want = [n for n, f in (("conv3d_fwd", 1), ("conv3d_wgrad", 2), ("colsum", 4)) if mask & f]
        else:
            want = [n for n, f in (("conv3d_dgrad", 1), ("conv3d_wgrad+db" if mask & 4 else "conv3d_wgrad", 2))
                    if mask & f]
            if mask & 4 and not mask & 2:
                want.append("colsum")
        assert log == want, (mask, log)
        stub.ms_record_free(h)
    assert stub.ms_testing_live_records() == 0


def test_conv3d_validation(stub):
    def fwd(a, x=None, W=None, y=None):
        h = ctypes.c_void_p()
        stub.stub_reset()
        st = stub.ms_layer_forward(ctypes.byref(a.layer), ref(x or a.x), ref(W or a.W), ref(a.b), 7,
                                   ref(y or a.y), ctypes.byref(h), None)
        assert stub.stub_log().decode() == "" and not h.value
        return st

    a = Conv3dArgs((2, 8, 6, 7, 5), 16, (3, 3, 3), (1, 1, 1), (1, 1, 1))
    assert fwd(a, x=tdesc(a.x_shape, layout="ncdhw")) == L.MS_E_LAYOUT
    assert fwd(a, W=tdesc((16, 8, 3, 3, 2))) == L.MS_E_SHAPE       # y no longer matches
    assert fwd(a, W=tdesc((16, 4, 3, 3, 3))) == L.MS_E_SHAPE
    assert fwd(a, x=tdesc((2, 8, 6, 7))) == L.MS_E_SHAPE            # 4-D x
    a.layer.stride_d = 0
    assert fwd(a) == L.MS_E_ARG
    a.layer.stride_d = 1
    a.layer.pad_d = -1
    assert fwd(a) == L.MS_E_ARG
    a.layer.pad_d = 1
    t = Conv3dArgs((2, 16, 3, 4, 4), 8, (2, 4, 4), (2, 2, 2), (0, 1, 1), (1, 0, 1))
    t.layer.out_pad_d = 2                                           # out_pad >= stride
    assert fwd(t) == L.MS_E_ARG


def test_output_size_limits_hold_for_extreme_padding(stub):
    """Pads near 2^30 make output extents near 2^31: the element-count
    checks must reject them (a plain int64 product of the extents would
    overflow) for the accounting call, which takes no y."""
    big = 1 << 30
    layer = L.MsLayer()
    layer.kind = L.MS_CONV2D
    layer.stride[0] = layer.stride[1] = 1
    layer.pad[0] = layer.pad[1] = big - 1
    x, w = tdesc((1, 1, 1, 1), data=False), tdesc((3, 1, 1, 1), data=False)
    a = L.MsAccount()
    assert stub.ms_policy_account(ctypes.byref(layer), ref(x), ref(w), None, 1, 0, ctypes.byref(a)) == L.MS_E_UNSUPPORTED
    l3 = L.MsLayer()
    l3.kind = L.MS_CONV3D
    l3.stride_d = l3.stride[0] = l3.stride[1] = 1
    l3.pad_d = l3.pad[0] = l3.pad[1] = big - 1
    x3, w3 = tdesc((1, 1, 1, 1, 1), data=False), tdesc((2, 1, 1, 1, 1), data=False)
    assert stub.ms_policy_account(ctypes.byref(l3), ref(x3), ref(w3), None, 1, 0, ctypes.byref(a)) == L.MS_E_UNSUPPORTED
