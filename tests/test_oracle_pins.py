"""Pins of the CPU oracle to the paper's worked examples and closed forms.

Each fixture under tests/golden/ carries the passage it comes from.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _one_head(q, K, V):
    """Wrap single-head arrays as B=1, h=1 batches."""
    q = np.asarray(q, np.float32).reshape(1, 1, -1)
    K = np.ascontiguousarray(np.asarray(K, np.float32)[None, None])
    V = np.ascontiguousarray(np.asarray(V, np.float32)[None, None])
    lens = np.array([K.shape[2]], np.int32)
    return q, K, V, lens


def test_worked_decode_example_matches_printed_values():
    """Decode DNF worked example: a ~ (0.670, 0.330), out ~ (3.32, 5.32)."""
    g = _golden("worked_decode_example.json")
    q, K, V, lens = _one_head(g["inputs"]["q"], g["inputs"]["K"], g["inputs"]["V"])
    scale = np.float32(1.0 / math.sqrt(2.0))
    w, row = oracle.decode_weights(q, K, V, lens, scale, 0, 0)
    out = oracle.decode(q, K, V, lens, scale)[0, 0]
    p, dec = g["printed"], g["printed_decimals"]
    half = lambda k: 0.5 * 10.0 ** (-dec[k]) + 1e-12
    assert np.all(np.abs(w - np.array(p["a"])) <= half("a"))
    assert np.all(np.abs(out - np.array(p["out"])) <= half("out"))
    assert np.array_equal(out, row)
    # e[1] and Z of Step II, from the weights: e = a / a[0] (e[0] = exp(0) = 1)
    e1 = w[1] / w[0]
    assert abs(e1 - p["e"][1]) <= half("e")
    assert abs(1.0 / w[0] - p["Z"]) <= half("Z")


def test_worked_decode_example_closed_form():
    """Closed form of the same example: with s = (c, 0), c = scale,
    a0 = 1 / (1 + e^{-c}) and out = a0*V[0] + (1-a0)*V[1]."""
    q, K, V, lens = _one_head([1, 0], [[1, 0], [0, 1]], [[2, 4], [6, 8]])
    scale = np.float32(1.0 / math.sqrt(2.0))
    c = float(scale)
    a0 = 1.0 / (1.0 + math.exp(-c))
    expect = np.array([2 * a0 + 6 * (1 - a0), 4 * a0 + 8 * (1 - a0)])
    out = oracle.decode(q, K, V, lens, scale)[0, 0]
    assert np.max(np.abs(out - expect)) <= 4e-15


def test_gamma_offsets_are_the_layout_both_sides_read():
    """ONF worked example: element <l,j> of a <3,2> slab is at l*2+j.  The
    arrays handed to the oracle and to the HIP library are C-contiguous, whose
    flat offsets must be exactly these."""
    g = _golden("gamma_example.json")
    shape = tuple(g["shape"])
    for key, off in g["offsets"].items():
        l, j = (int(x) for x in key.split(","))
        assert np.ravel_multi_index((l, j), shape) == off
    # And the oracle reads K by those offsets: a <3,2> slab whose rows are
    # told apart only by column 1 (flat offsets 1, 3, 5).
    flat = np.array([5, 0, 0, 5, 1, 1], np.float32)
    K = flat.reshape(3, 2)
    V = np.array([[1, 0], [0, 1], [7, 7]], np.float32)
    q, Kb, Vb, lens = _one_head([0, 1], K, V)
    out = oracle.decode(q, Kb, Vb, lens, np.float32(200.0))[0, 0]
    # row 1 (offsets 2,3) has K[1,1]=5: the others trail by >= 800 and
    # underflow to exactly zero weight in fp64
    assert np.array_equal(out, np.array([0.0, 1.0]))


def test_append_example_writes_offsets_6_7_8_only():
    """Cache-append worked example: t=2, d_k=3, new row at offsets 6, 7, 8,
    no existing element moved."""
    g = _golden("append_example.json")
    t, d_k = g["t"], g["d_k"]
    n_max = 5
    K = np.arange(n_max * d_k, dtype=np.float32).reshape(1, 1, n_max, d_k) + 100
    V = np.zeros((1, 1, n_max, 1), np.float32)
    before = K.copy()
    lens = np.array([t], np.int32)
    k_new = np.array([[[-1.0, -2.0, -3.0]]], np.float32)
    oracle.append(K, V, k_new, np.zeros((1, 1, 1), np.float32), lens)
    flat, flat0 = K.reshape(-1), before.reshape(-1)
    changed = np.nonzero(flat != flat0)[0].tolist()
    assert changed == g["new_row_offsets"]
    assert flat[changed].tolist() == [-1.0, -2.0, -3.0]
    assert lens[0] == t + 1


def test_append_at_capacity_is_a_no_op():
    K = np.zeros((1, 2, 3, 4), np.float32)
    V = np.zeros((1, 2, 3, 4), np.float32)
    lens = np.array([3], np.int32)
    oracle.append(K, V, np.ones((1, 2, 4), np.float32),
                  np.ones((1, 2, 4), np.float32), lens)
    assert lens[0] == 3 and not K.any() and not V.any()


@pytest.mark.parametrize("case", _golden("gqa_head_map.json")["cases"])
def test_gqa_head_map(case):
    """psi-selection: query head h reads KV slab floor(h*h_kv/h_q).  Make
    every V slab constant = its index; the output of head h is that index."""
    h_q, h_kv = case["h_q"], case["h_kv"]
    n, d = 3, 2
    rng = np.random.default_rng(7)
    q = rng.standard_normal((1, h_q, d)).astype(np.float32)
    K = rng.standard_normal((1, h_kv, n, d)).astype(np.float32)
    V = np.empty((1, h_kv, n, d), np.float32)
    for g in range(h_kv):
        V[0, g] = g
    out = oracle.decode(q, K, V, np.array([n], np.int32), np.float32(0.7))
    got = [int(round(out[0, h, 0])) for h in range(h_q)]
    assert got == case["kv_head_of"]
    assert np.max(np.abs(out[0, :, 0] - np.array(case["kv_head_of"]))) < 1e-14


def test_empty_cache_gives_zero():
    q = np.ones((2, 2, 4), np.float32)
    K = np.full((2, 1, 3, 4), np.nan, np.float32)
    V = np.full((2, 1, 3, 4), np.nan, np.float32)
    out = oracle.decode(q, K, V, np.array([0, 0], np.int32), np.float32(0.5))
    assert np.array_equal(out, np.zeros((2, 2, 4)))


def test_rows_beyond_len_are_not_read():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 8)).astype(np.float32)
    K = rng.standard_normal((1, 1, 6, 8)).astype(np.float32)
    V = rng.standard_normal((1, 1, 6, 8)).astype(np.float32)
    ref = oracle.decode(q, K, V, np.array([4], np.int32), np.float32(0.3))
    K[0, 0, 4:] = np.nan
    V[0, 0, 4:] = np.inf
    out = oracle.decode(q, K, V, np.array([4], np.int32), np.float32(0.3))
    assert np.array_equal(out, ref)


def test_len_beyond_capacity_is_clamped():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 1, 8)).astype(np.float32)
    K = rng.standard_normal((1, 1, 6, 8)).astype(np.float32)
    V = rng.standard_normal((1, 1, 6, 8)).astype(np.float32)
    a = oracle.decode(q, K, V, np.array([6], np.int32), np.float32(0.3))
    b = oracle.decode(q, K, V, np.array([1000], np.int32), np.float32(0.3))
    assert np.array_equal(a, b)


def test_shape_errors_are_rejected():
    q = np.ones((1, 3, 4), np.float32)
    K = np.ones((1, 2, 3, 4), np.float32)
    with pytest.raises(ValueError):
        oracle.decode(q, K, K, np.array([3], np.int32), np.float32(1))
