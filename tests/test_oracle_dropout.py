"""Pins of the dropout oracle (Sec. 2.2.2: keep the generator state, draw
the mask again in backward): the published Philox4x32-10 known-answer
vectors, keep decisions derived by hand from them, the layout of the stream
over elements, the statistics of the draw, the special cases p = 0 and
p = 1, and linearity / the adjoint identity of the forward map."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import policy as P

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")))


def _h(words):
    return [int(w, 16) for w in words]


@pytest.mark.parametrize("i", range(len(GOLD["vectors"])))
def test_philox_known_answers(i):
    v = GOLD["vectors"][i]
    assert oracle.philox4x32_10(_h(v["ctr"]), _h(v["key"])).tolist() == _h(v["out"])


@pytest.mark.parametrize("i", range(len(GOLD["dropout_cases"])))
def test_keep_decisions_worked_by_hand(i):
    c = GOLD["dropout_cases"][i]
    assert oracle.dropout_keep(4, c["p"], c["seed"], c["offset"]).tolist() == c["keep"]


def test_first_block_is_the_first_known_answer():
    """Seed 0, offset 0: elements 0..3 take the words of counter 0, key 0."""
    assert oracle.dropout_words(4, 0, 0).tolist() == _h(GOLD["vectors"][0]["out"])


def test_stream_layout_over_elements_and_counter_words():
    seed = 0x123456789ABCDEF0
    u = oracle.dropout_words(40, seed, 7)
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for blk in range(10):
        assert u[4 * blk:4 * blk + 4].tolist() == oracle.philox4x32_10([7 + blk, 0, 0, 0], key).tolist()
    # an offset past 2^32 carries into the second counter word
    off = (5 << 32) + 0xFFFFFFFE
    u = oracle.dropout_words(12, seed, off)
    assert u[0:4].tolist() == oracle.philox4x32_10([0xFFFFFFFE, 5, 0, 0], key).tolist()
    assert u[8:12].tolist() == oracle.philox4x32_10([0, 6, 0, 0], key).tolist()
    # a ragged tail takes the leading words of its block
    assert oracle.dropout_words(10, seed, 7).tolist() == oracle.dropout_words(12, seed, 7)[:10].tolist()
    # shifting the offset by k blocks drops the first 4k words
    assert oracle.dropout_words(36, seed, 9).tolist() == oracle.dropout_words(44, seed, 7)[8:].tolist()


@pytest.mark.parametrize("p", [0.1, 0.5, 0.9])
def test_keep_fraction_is_binomial(p):
    n = 1 << 20
    k = int(oracle.dropout_keep(n, p, 20240417, 3).sum())
    mean, sd = n * (1 - p), math.sqrt(n * p * (1 - p))
    assert abs(k - mean) < 5 * sd


def test_words_are_uniform_and_adjacent_keeps_uncorrelated():
    u = oracle.dropout_words(1 << 20, 99, 0)
    counts = np.bincount(u >> 24, minlength=256)
    exp = u.size / 256
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 255 + 6 * math.sqrt(2 * 255)
    keep = (u >= np.uint32(1 << 31)).astype(np.float64)
    r = np.corrcoef(keep[:-1], keep[1:])[0, 1]
    assert abs(r) < 5 / math.sqrt(u.size)


def test_seeds_and_offsets_give_different_masks():
    a = oracle.dropout_keep(4096, 0.5, 1, 0)
    assert (a != oracle.dropout_keep(4096, 0.5, 2, 0)).mean() > 0.4
    assert (a != oracle.dropout_keep(4096, 0.5, 1, 1024)).mean() > 0.4
    assert (a != oracle.dropout_keep(4096, 0.5, 1 << 32, 0)).mean() > 0.4   # the key's high word counts


def test_threshold_and_scale():
    assert oracle.dropout_threshold(0.0) == (0, False)
    assert oracle.dropout_threshold(1.0) == (0, True)
    assert oracle.dropout_threshold(0.5) == (1 << 31, False)
    assert oracle.dropout_scale(0.5) == 2.0
    assert oracle.dropout_scale(0.2) == float(np.float32(1.0 / (1.0 - float(np.float32(0.2)))))
    with pytest.raises(ValueError):
        oracle.dropout_threshold(1.5)


def test_special_cases():
    x = np.random.default_rng(0).standard_normal(1001)
    np.testing.assert_array_equal(oracle.dropout_forward(x, 0.0, 5), x)
    np.testing.assert_array_equal(oracle.dropout_forward(x, 1.0, 5), np.zeros_like(x))
    y = oracle.dropout_forward(x, 0.5, 5)
    keep = oracle.dropout_keep(x.size, 0.5, 5)
    np.testing.assert_array_equal(y[keep], 2.0 * x[keep])
    assert np.all(y[~keep] == 0.0)


def test_linear_map_and_its_adjoint():
    rng = np.random.default_rng(1)
    x1, x2, dy = rng.standard_normal((3, 777))
    y = lambda v: oracle.dropout_forward(v, 0.3, 11, 2)
    np.testing.assert_allclose(y(2.0 * x1 - 3.0 * x2), 2.0 * y(x1) - 3.0 * y(x2), rtol=1e-14, atol=1e-14)
    assert np.isclose(np.vdot(y(x1), dy), np.vdot(x1, oracle.dropout_backward(dy, 0.3, 11, 2)), rtol=1e-13)


def test_policy_closed_form():
    n = 1000
    assert P.saved_activation_bytes("dropout", 1, n, "bf16", P.SELECTIVE) == 0
    assert P.saved_activation_bytes("dropout", 1, n, "bf16", P.PYTORCH_DEFAULT) == n
    assert P.saved_activation_bytes("dropout", 0, n, "bf16", P.PYTORCH_DEFAULT) == 0
    assert P.launched("dropout", 1) == {"dgrad": True, "wgrad": False, "bgrad": False}
