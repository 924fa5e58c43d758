"""Invariants the decode attention result must satisfy, checked on the oracle.

Inputs use small dyadic values where an invariant needs exact fp32 inputs
(shifted keys, linear combinations of V), so the only rounding is the
oracle's own fp64 arithmetic.
"""
import numpy as np
import pytest

import oracle


def _dyadic(rng, shape, lo=-16, hi=16, denom=8.0):
    return (rng.integers(lo, hi, size=shape) / denom).astype(np.float32)


def _case(seed, B=2, h_q=4, h_kv=2, n_max=9, d_k=6, d_v=5):
    rng = np.random.default_rng(seed)
    q = _dyadic(rng, (B, h_q, d_k))
    K = _dyadic(rng, (B, h_kv, n_max, d_k))
    V = _dyadic(rng, (B, h_kv, n_max, d_v))
    lens = rng.integers(1, n_max + 1, size=B).astype(np.int32)
    return q, K, V, lens


@pytest.mark.parametrize("seed", range(4))
def test_weights_sum_to_one(seed):
    q, K, V, lens = _case(seed)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            w, _ = oracle.decode_weights(q, K, V, lens, np.float32(0.4), b, h)
            assert len(w) == lens[b]
            assert np.all(w >= 0)
            assert abs(w.sum() - 1.0) <= 1e-14


def test_single_row_returns_that_row_exactly():
    q, K, V, _ = _case(5)
    lens = np.array([1, 1], np.int32)
    out = oracle.decode(q, K, V, lens, np.float32(0.3))
    for b in range(2):
        for h in range(4):
            assert np.array_equal(out[b, h], V[b, h // 2, 0].astype(np.float64))


def test_identical_keys_return_mean_of_v():
    q, K, V, lens = _case(6)
    K[:] = K[:, :, :1, :]          # every row equals row 0
    out = oracle.decode(q, K, V, lens, np.float32(0.3))
    for b in range(2):
        n = lens[b]
        for h in range(4):
            mean = V[b, h // 2, :n].astype(np.float64).mean(axis=0)
            assert np.max(np.abs(out[b, h] - mean)) <= 1e-14


def test_zero_scale_returns_mean_of_v():
    q, K, V, lens = _case(7)
    out = oracle.decode(q, K, V, lens, np.float32(0.0))
    for b in range(2):
        for h in range(4):
            mean = V[b, h // 2, :lens[b]].astype(np.float64).mean(axis=0)
            assert np.max(np.abs(out[b, h] - mean)) <= 1e-14


@pytest.mark.parametrize("h_kv", [1, 2, 4, 8])
def test_gqa_equals_mha_with_repeated_kv(h_kv):
    rng = np.random.default_rng(h_kv)
    h_q, G = 8, 8 // h_kv
    q = rng.standard_normal((2, h_q, 8)).astype(np.float32)
    K = rng.standard_normal((2, h_kv, 10, 8)).astype(np.float32)
    V = rng.standard_normal((2, h_kv, 10, 4)).astype(np.float32)
    lens = np.array([10, 7], np.int32)
    gqa = oracle.decode(q, K, V, lens, np.float32(0.35))
    Kx = np.ascontiguousarray(np.repeat(K, G, axis=1))
    Vx = np.ascontiguousarray(np.repeat(V, G, axis=1))
    mha = oracle.decode(q, Kx, Vx, lens, np.float32(0.35))
    assert np.array_equal(gqa, mha)


def test_append_then_decode_equals_decode_on_full_cache():
    rng = np.random.default_rng(9)
    B, h_kv, h_q, n_max, d = 2, 2, 4, 12, 8
    full_K = rng.standard_normal((B, h_kv, n_max, d)).astype(np.float32)
    full_V = rng.standard_normal((B, h_kv, n_max, d)).astype(np.float32)
    start = np.array([5, 8], np.int32)
    K = np.full_like(full_K, np.nan)
    V = np.full_like(full_V, np.nan)
    for b in range(B):
        K[b, :, :start[b]] = full_K[b, :, :start[b]]
        V[b, :, :start[b]] = full_V[b, :, :start[b]]
    lens = start.copy()
    for step in range(3):
        kn = np.ascontiguousarray(full_K[np.arange(B), :, lens])  # [B, h_kv, d]
        vn = np.ascontiguousarray(full_V[np.arange(B), :, lens])
        oracle.append(K, V, kn, vn, lens)
        q = rng.standard_normal((B, h_q, d)).astype(np.float32)
        got = oracle.decode(q, K, V, lens, np.float32(0.3))
        ref = oracle.decode(q, full_K, full_V, lens, np.float32(0.3))
        assert np.array_equal(got, ref)
        assert lens.tolist() == (start + step + 1).tolist()


def test_row_permutation_leaves_output_unchanged():
    q, K, V, _ = _case(10, n_max=9)
    lens = np.array([9, 9], np.int32)
    perm = np.random.default_rng(1).permutation(9)
    a = oracle.decode(q, K, V, lens, np.float32(0.4))
    b = oracle.decode(q, np.ascontiguousarray(K[:, :, perm]),
                      np.ascontiguousarray(V[:, :, perm]), lens, np.float32(0.4))
    assert np.max(np.abs(a - b)) <= 1e-14


def test_shifting_every_key_by_one_vector_leaves_output_unchanged():
    """s_l -> s_l + scale*q.c for all l: softmax is shift-invariant."""
    q, K, V, lens = _case(11)
    c = _dyadic(np.random.default_rng(2), (1, 1, 1, K.shape[3]))
    K2 = (K + c).astype(np.float32)
    assert np.array_equal(K2.astype(np.float64), K.astype(np.float64) + c)
    a = oracle.decode(q, K, V, lens, np.float32(0.25))
    b = oracle.decode(q, K2, V, lens, np.float32(0.25))
    assert np.max(np.abs(a - b)) <= 1e-13


def test_output_is_linear_in_v():
    q, K, V1, lens = _case(12)
    V2 = _dyadic(np.random.default_rng(3), V1.shape)
    Vc = (2 * V1 - 3 * V2).astype(np.float32)
    assert np.array_equal(Vc.astype(np.float64), 2.0 * V1 - 3.0 * V2)
    o1 = oracle.decode(q, K, V1, lens, np.float32(0.5))
    o2 = oracle.decode(q, K, V2, lens, np.float32(0.5))
    oc = oracle.decode(q, K, Vc, lens, np.float32(0.5))
    assert np.max(np.abs(oc - (2 * o1 - 3 * o2))) <= 1e-13


def test_one_dominant_key_selects_its_value_row():
    rng = np.random.default_rng(13)
    q = rng.standard_normal((1, 1, 8)).astype(np.float32)
    K = (0.01 * rng.standard_normal((1, 1, 20, 8))).astype(np.float32)
    K[0, 0, 13] = q[0, 0] * 4
    V = rng.standard_normal((1, 1, 20, 8)).astype(np.float32)
    out = oracle.decode(q, K, V, np.array([20], np.int32), np.float32(100.0))
    assert np.max(np.abs(out[0, 0] - V[0, 0, 13])) <= 1e-12


def test_result_is_a_convex_combination_of_value_rows():
    q, K, V, lens = _case(14)
    out = oracle.decode(q, K, V, lens, np.float32(0.7))
    for b in range(2):
        for h in range(4):
            rows = V[b, h // 2, :lens[b]]
            assert np.all(out[b, h] <= rows.max(axis=0) + 1e-14)
            assert np.all(out[b, h] >= rows.min(axis=0) - 1e-14)
