"""The bf16 GEMM planner's decisions, queried through the library's testing
hook (no GPU: planning is host code).  Pins the choices the measured
headline relies on and checks the invariants of the column split and of the
tiles that exist only for some contractions."""
import ctypes
import itertools

import pytest

from paper_2404_12406_amd import _lib

G = ctypes.c_int32 * 13
O = ctypes.c_int32 * 10
FWD, DGRAD, WGRAD = 0, 1, 2


@pytest.fixture(scope="module")
def lib():
    return _lib.configure(ctypes.CDLL(_lib.LIB_PATH))


def plan(lib, pas, geom):
    o = O()
    r = lib.ms_testing_gemm_plan(pas, G(*geom), o)
    keys = ("bm", "bn", "waves", "stages", "kg", "splits", "direct", "n1", "bm2", "bn2")
    return r, dict(zip(keys, list(o)))


def linear(M, k_in, n_out):
    # a Linear layer is the 1x1 convolution over M "images" of 1 x 1 pixels
    return (M, k_in, 1, 1, n_out, 1, 1, 1, 1, 1, 1, 0, 0)


def tiles(M, N, bm, bn):
    return -(-M // bm) * -(-N // bn)


def test_headline_shapes(lib):
    """The encoder linears at 8192 tokens: the QKV forward takes the 256 x 288
    tile (256 tiles, one wave); the forward of FFN up and the input gradient
    of FFN down split their output columns at 2048 (256 tiles of 256 x 256,
    one per CU) and cover the rest on a second tile; the 768-wide outputs
    take the 128 x 192 tile (256 tiles, one wave)."""
    r, p = plan(lib, FWD, linear(8192, 768, 2304))
    assert r == 0 and (p["bm"], p["bn"], p["n1"]) == (256, 288, 0) and p["splits"] == 1
    assert tiles(8192, 2304, 256, 288) == 256
    r, p = plan(lib, FWD, linear(8192, 768, 3072))
    assert r == 0 and (p["bm"], p["bn"], p["n1"], p["bm2"], p["bn2"]) == (256, 256, 2048, 256, 128)
    r, p = plan(lib, DGRAD, linear(8192, 3072, 768))
    assert r == 0 and (p["bm"], p["bn"], p["n1"], p["bm2"], p["bn2"]) == (256, 256, 2048, 256, 128)
    assert p["direct"] == 1
    for shape in (linear(8192, 768, 768), linear(8192, 3072, 768)):
        r, p = plan(lib, FWD, shape)
        assert r == 0 and (p["bm"], p["bn"], p["n1"]) == (128, 192, 0)
        assert tiles(8192, 768, 128, 192) == 256


def _sweep():
    Ms = (300, 4096, 6000, 8192, 12800)
    widths = (64, 136, 768, 1032, 2304, 3072, 4200)
    return itertools.product(Ms, widths, widths)


@pytest.mark.parametrize("pas", [FWD, DGRAD])
def test_column_split_invariants(lib, pas):
    """Wherever a column split is taken: one split only, the first launch's
    columns are whole tile columns short of the output width, as many as fit
    in the whole waves of 256 CUs that the first plan's tiles fill, and those
    tiles would have left a partial last wave."""
    seen = 0
    for M, k_in, n_out in _sweep():
        r, p = plan(lib, pas, linear(M, k_in, n_out))
        assert r == 0
        if p["n1"] == 0:
            continue
        seen += 1
        width = n_out if pas == FWD else k_in
        assert p["splits"] == 1
        assert 0 < p["n1"] < width and p["n1"] % p["bn"] == 0
        ntm = -(-M // p["bm"])
        first = tiles(M, p["n1"], p["bm"], p["bn"])
        total = tiles(M, width, p["bm"], p["bn"])
        whole = total // 256 * 256          # one block per CU on the tiles that split
        assert total % 256 != 0 and whole - ntm < first <= whole, (M, k_in, n_out, p)
        assert p["bm2"] > 0 and p["bn2"] > 0
    assert seen > 0


def test_column_split_knob(lib, monkeypatch):
    """MEMSAVE_GEMM_TAIL=off never splits; =on splits wherever the first
    plan's tiles leave a partial last wave of one-block-per-CU tiles."""
    monkeypatch.setenv("MEMSAVE_GEMM_TAIL", "off")
    for M, k_in, n_out in _sweep():
        for pas in (FWD, DGRAD):
            assert plan(lib, pas, linear(M, k_in, n_out))[1]["n1"] == 0
    monkeypatch.setenv("MEMSAVE_GEMM_TAIL", "on")
    r, p = plan(lib, FWD, linear(8192, 64, 3072))
    assert r == 0 and (p["bm"], p["bn"]) == (256, 256) and p["n1"] == 2048
    monkeypatch.setenv("MEMSAVE_GEMM_TILE", "256x128")
    assert plan(lib, FWD, linear(8192, 768, 3072))[1]["n1"] == 0   # a forced tile is never split


def test_tiles_that_exist_for_some_contractions_only(lib):
    """The 192-wide and 32-wide tiles read both operands k-contiguous: never
    for an input gradient that reads W in place, and the 192-wide one only
    where it fills the CUs in one wave; a strided input gradient always goes
    through the transposed filter."""
    for M, k_in, n_out in _sweep():
        r, p = plan(lib, FWD, linear(M, k_in, n_out))
        if p["bn"] == 192:
            assert tiles(M, n_out, 128, 192) <= 256
        if p["bn"] == 288:
            assert tiles(M, n_out, 256, 288) <= 256
        r, p = plan(lib, DGRAD, linear(M, k_in, n_out))
        assert p["bn"] != 288   # the 288-wide tile is built for the forward only
        if p["direct"]:
            assert p["bn"] not in (32, 192)
        if p["bn"] == 192:
            assert tiles(M, k_in, 128, 192) <= 256
    conv_s2 = (64, 64, 56, 56, 128, 3, 3, 28, 28, 2, 2, 1, 1)
    r, p = plan(lib, DGRAD, conv_s2)
    assert r == 0 and p["direct"] == 0 and p["n1"] == 0



def test_forced_288_tile_only_where_built(lib, monkeypatch):
    """MEMSAVE_GEMM_TILE=256x288 is honoured by the Linear (1x1) forward only;
    a convolution forward, an input gradient and a weight gradient plan as if
    it were not forced."""
    monkeypatch.setenv("MEMSAVE_GEMM_TILE", "256x288")
    r, p = plan(lib, FWD, linear(4096, 512, 1000))
    assert r == 0 and (p["bm"], p["bn"]) == (256, 288)
    assert plan(lib, FWD, conv(64, 64, 56, 128, 3, 2, 1))[1]["bn"] != 288
    assert plan(lib, DGRAD, linear(8192, 768, 2304))[1]["bn"] != 288
    assert plan(lib, WGRAD, linear(8192, 768, 2304))[1]["bn"] != 288


def test_weight_gradient_and_refusals(lib):
    r, p = plan(lib, WGRAD, (32, 256, 28, 28, 256, 3, 3, 28, 28, 1, 1, 1, 1))
    assert r == 0 and p["splits"] > 1 and p["kg"] == 1
    # channel counts that are not multiples of 8 are not the fast path's
    assert plan(lib, FWD, (64, 3, 224, 224, 64, 7, 7, 112, 112, 2, 2, 3, 3))[0] == -1


def conv(N, C, H, K, R, stride, pad):
    P = (H + 2 * pad - R) // stride + 1
    return (N, C, H, H, K, R, R, P, P, stride, stride, pad, pad)


def test_tap_step_convs_plan_without_k_groups(lib):
    """Convolutions whose reduction channels are a multiple of 64 (the
    forward's C, the input gradient's K) run on the tap-step operand loads
    and plan over the tiles without k-groups: the ResNet-18-shaped stage-3
    3x3 layer takes the 8-wave 4-stage 128 x 128 tile both ways, and no
    tap-step convolution of the stack or the sweep takes a k-group tile."""
    for pas in (FWD, DGRAD):
        r, p = plan(lib, pas, conv(64, 256, 14, 256, 3, 1, 1))
        assert r == 0 and (p["bm"], p["bn"], p["waves"], p["stages"], p["kg"]) == (128, 128, 8, 4, 1)
    shapes = [conv(64, 64, 56, 128, 3, 2, 1), conv(64, 128, 28, 128, 3, 1, 1), conv(64, 128, 28, 256, 3, 2, 1),
              conv(64, 256, 14, 512, 3, 2, 1), conv(64, 512, 7, 512, 3, 1, 1), conv(32, 256, 28, 256, 3, 1, 1)]
    for geom, pas in itertools.product(shapes, (FWD, DGRAD)):
        r, p = plan(lib, pas, geom)
        assert r == 0 and p["kg"] == 1, (geom, pas, p)


def test_conv_weight_gradient_splits_stay_in_one_wave(lib):
    """The convolution weight gradient prices its split reduction and tries
    every split count: the 3x3 sweep layer (256 x 2304 outputs, 36 tiles of
    128 x 128) takes 7 splits, 252 blocks in one wave of 256 CUs, where
    ceil(256 / 36) = 8 would spill 32 blocks into a second; no plan of the
    stack, the sweep or the decoder runs more blocks than one wave holds."""
    r, p = plan(lib, WGRAD, conv(32, 256, 28, 256, 3, 1, 1))
    assert r == 0 and (p["bm"], p["bn"], p["splits"]) == (128, 128, 7)
    shapes = [conv(32, 256, 28, 256, 3, 1, 1), conv(64, 128, 28, 128, 3, 1, 1), conv(64, 128, 28, 256, 3, 2, 1),
              conv(64, 512, 7, 512, 3, 1, 1), conv(64, 64, 56, 64, 3, 1, 1), conv(32, 128, 56, 256, 4, 2, 1)]
    for geom in shapes:
        r, p = plan(lib, WGRAD, geom)
        N, C, H, _, K, R, S = geom[:7]
        blocks = tiles(K, R * S * C, p["bm"], p["bn"]) * p["splits"]
        per_cu = 1 if p["stages"] == 4 or p["bm"] == 256 else 2
        assert r == 0 and blocks <= 256 * per_cu, (geom, p, blocks)
