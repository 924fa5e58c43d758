"""Pins of the oracle's multi-row (causal) decode and of the T-row append.

A step that submits T consecutive positions at once (speculative
verification, chunked prefill) is the paper's rank-2 query form,
softmax(scale * Q (+.x Omega<2,2>) K) (+.x Omega<2,2>) V, with causal
visibility: row r of sequence b sits at cache position len[b] - T + r and
sees rows 0 .. that position.  Pinned against
* PyTorch's SDPA in float64 with is_causal=True (the whole cache is the T
  rows) and with an explicit boolean mask (a cache longer than T), GQA by
  repeating KV heads -- the paper's own ground truth, a library routine;
* T single-query steps of the pinned decode and append (the multi-step KV
  cache of the paper's Section 5), which must give the same numbers bit for
  bit;
* a 50-digit ``decimal`` brute force on tiny shapes.
"""
import math
from decimal import Decimal, getcontext

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2607_19456_amd import workloads

getcontext().prec = 50


def _rand(seed, shape):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


def _sdpa_masked(q, K, V, lens, scale, causal_full=False):
    """q [B,h_q,T,d_k], K/V [B,h_kv,n_max,d]; float64 SDPA per sequence with
    KV heads repeated G times and the causal mask of the last T positions."""
    B, h_q, T, d_k = q.shape
    _, h_kv, n_max, _ = K.shape
    G = h_q // h_kv
    out = np.zeros(q.shape[:3] + (V.shape[3],))
    for b in range(B):
        n = min(max(int(lens[b]), 0), n_max)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).double()
        Kx = t(np.repeat(K[b, :, :n], G, axis=0))
        Vx = t(np.repeat(V[b, :, :n], G, axis=0))
        if causal_full:
            assert n == T
            o = F.scaled_dot_product_attention(t(q[b]), Kx, Vx, scale=float(scale),
                                               is_causal=True)
        else:
            pos = n - T + np.arange(T)
            allowed = torch.from_numpy(np.arange(n)[None, :] <= pos[:, None])
            o = F.scaled_dot_product_attention(t(q[b]), Kx, Vx, attn_mask=allowed,
                                               scale=float(scale))
        out[b] = o.numpy()
    return out


@pytest.mark.parametrize("T,d,h_q,h_kv", [(4, 8, 2, 2), (16, 64, 4, 1), (7, 32, 6, 3)])
def test_whole_cache_equals_causal_sdpa(T, d, h_q, h_kv):
    q = _rand([1, T, d], (2, h_q, T, d))
    K = _rand([2, T, d], (2, h_kv, T, d))
    V = _rand([3, T, d], (2, h_kv, T, d))
    scale = np.float32(1 / math.sqrt(d))
    lens = np.array([T, T], np.int32)
    got = oracle.decode_multi(q, K, V, lens, scale)
    ref = _sdpa_masked(q, K, V, lens, scale, causal_full=True)
    assert np.max(np.abs(got - ref)) <= 1e-12


@pytest.mark.parametrize("T,lens", [(4, [37, 9]), (3, [5, 64]), (8, [8, 40])])
def test_longer_cache_equals_masked_sdpa(T, lens):
    d, h_q, h_kv, n_max = 16, 8, 2, 64
    q = _rand([4, T], (2, h_q, T, d))
    K = _rand([5, T], (2, h_kv, n_max, d))
    V = _rand([6, T], (2, h_kv, n_max, d))
    scale = np.float32(0.3)
    lens = np.array(lens, np.int32)
    got = oracle.decode_multi(q, K, V, lens, scale)
    ref = _sdpa_masked(q, K, V, lens, scale)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_equals_t_single_steps_bit_for_bit():
    """append_rows + decode_multi == T x (append one row, decode its query)."""
    B, h_q, h_kv, n_max, d_k, d_v, T = 3, 8, 2, 50, 16, 8, 5
    shape = workloads.custom("multi_seq", B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v,
                             n_max=n_max)
    inp = workloads.make(shape, seed=2, lens=np.array([0, 20, 44], np.int32))
    kn = _rand(7, (B, h_kv, T, d_k))
    vn = _rand(8, (B, h_kv, T, d_v))
    q = _rand(9, (B, h_q, T, d_k))
    # sequential: the pinned single-row path
    K1, V1, l1 = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    seq = np.zeros((B, h_q, T, d_v))
    for r in range(T):
        oracle.append(K1, V1, np.ascontiguousarray(kn[:, :, r]),
                      np.ascontiguousarray(vn[:, :, r]), l1)
        seq[:, :, r] = oracle.decode(np.ascontiguousarray(q[:, :, r]), K1, V1, l1, 0.25)
    # the chunk: T rows at once
    K2, V2, l2 = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    oracle.append_rows(K2, V2, kn, vn, l2)
    chunk = oracle.decode_multi(q, K2, V2, l2, 0.25)
    assert l2.tolist() == l1.tolist() == [5, 25, 49]
    assert np.array_equal(K1.view(np.uint32), K2.view(np.uint32))
    assert np.array_equal(V1.view(np.uint32), V2.view(np.uint32))
    assert np.array_equal(seq, chunk)


def test_near_capacity_the_two_multi_row_forms_differ_as_documented():
    """T single steps (what the fused multi-row step computes) and append_rows
    + decode_multi coincide only while every row fits.  With len = n_max - 2
    and T = 4, single step r attends min(len + r + 1, n_max) rows, the
    multi-row decode's row r attends n_max - T + r + 1 rows (the cache's last
    T positions); a full cache (len = n_max) appends nothing and both then
    attend n_max - T + r + 1 ... n_max rows differently again."""
    B, h_q, h_kv, n_max, d, T = 2, 4, 2, 40, 8, 4
    shape = workloads.custom("near_cap_o", B=B, h_q=h_q, h_kv=h_kv, d_k=d, d_v=d,
                             n_max=n_max)
    inp = workloads.make(shape, seed=3, lens=np.array([n_max - 2, n_max], np.int32))
    kn, vn, q = _rand(20, (B, h_kv, T, d)), _rand(21, (B, h_kv, T, d)), _rand(22, (B, h_q, T, d))
    K1, V1, l1 = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    seq = np.zeros((B, h_q, T, d))
    for r in range(T):
        oracle.append(K1, V1, np.ascontiguousarray(kn[:, :, r]),
                      np.ascontiguousarray(vn[:, :, r]), l1)
        seq[:, :, r] = oracle.decode(np.ascontiguousarray(q[:, :, r]), K1, V1, l1, 0.25)
    K2, V2, l2 = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    oracle.append_rows(K2, V2, kn, vn, l2)
    multi = oracle.decode_multi(q, K2, V2, l2, 0.25)
    assert l1.tolist() == l2.tolist() == [n_max, n_max]
    assert np.array_equal(K1.view(np.uint32), K2.view(np.uint32))
    for r in range(T):
        qr = np.ascontiguousarray(q[:, :, r])
        seq_rows = np.minimum(inp.lens + r + 1, n_max).astype(np.int32)
        multi_rows = np.full(B, n_max - T + r + 1, np.int32)
        assert np.array_equal(seq[:, :, r], oracle.decode(qr, K1, V1, seq_rows, 0.25))
        assert np.array_equal(multi[:, :, r], oracle.decode(qr, K1, V1, multi_rows, 0.25))
    # the rows whose visibility differs give different outputs
    assert not np.allclose(seq[0, :, 0], multi[0, :, 0])      # n_max-1 vs n_max-3 rows
    assert np.array_equal(seq[0, :, 3], multi[0, :, 3])       # both see the whole cache
    assert not np.allclose(seq[1, :, 0], multi[1, :, 0])      # full cache: n_max vs n_max-3


def test_one_row_is_the_single_query_decode():
    q = _rand(10, (2, 4, 1, 8))
    K = _rand(11, (2, 2, 30, 8))
    V = _rand(12, (2, 2, 30, 8))
    lens = np.array([30, 3], np.int32)
    a = oracle.decode_multi(q, K, V, lens, 0.5)[:, :, 0]
    b = oracle.decode(np.ascontiguousarray(q[:, :, 0]), K, V, lens, 0.5)
    assert np.array_equal(a, b)


def test_rows_before_the_cache_start_are_zero():
    """len < T: the first T - len rows have no visible key (position < 0)."""
    T = 6
    q = _rand(13, (1, 2, T, 4))
    K = _rand(14, (1, 1, 10, 4))
    V = _rand(15, (1, 1, 10, 4))
    out = oracle.decode_multi(q, K, V, np.array([2], np.int32), 1.0)
    assert np.array_equal(out[0, :, :4], np.zeros((2, 4, 4)))
    # row T-1 sees rows 0..1, row T-2 sees row 0 only: that row's V exactly
    assert np.array_equal(out[0, 0, T - 2], V[0, 0, 0].astype(np.float64))
    assert np.all(np.isfinite(out))


def test_last_row_sees_the_whole_cache_and_first_row_is_causal():
    q = _rand(16, (1, 1, 3, 8))
    K = _rand(17, (1, 1, 12, 8))
    V = _rand(18, (1, 1, 12, 8))
    out = oracle.decode_multi(q, K, V, np.array([12], np.int32), 0.4)
    full = oracle.decode(np.ascontiguousarray(q[:, :, 2]), K, V, np.array([12], np.int32), 0.4)
    first = oracle.decode(np.ascontiguousarray(q[:, :, 0]), K, V, np.array([10], np.int32), 0.4)
    assert np.array_equal(out[:, :, 2], full)
    assert np.array_equal(out[:, :, 0], first)
    # rows of the cache beyond a row's position must not matter
    K2 = K.copy()
    K2[0, 0, 10:] = np.nan
    out2 = oracle.decode_multi(q, K2, V, np.array([12], np.int32), 0.4)
    assert np.array_equal(out2[:, :, 0], out[:, :, 0])


def _brute_multi(q, K, V, lens, scale):
    B, h_q, T, d_k = q.shape
    _, h_kv, n_max, _ = K.shape
    G = h_q // h_kv
    sc = Decimal(float(np.float32(scale)))
    out = np.zeros((B, h_q, T, V.shape[3]))
    for b in range(B):
        n = min(max(int(lens[b]), 0), n_max)
        for h in range(h_q):
            g = h // G
            for r in range(T):
                vis = [l for l in range(n) if l <= n - T + r]
                if not vis:
                    continue
                ex = [(sc * sum(Decimal(float(q[b, h, r, j])) * Decimal(float(K[b, g, l, j]))
                                for j in range(d_k))).exp() for l in vis]
                Z = sum(ex)
                for d in range(V.shape[3]):
                    out[b, h, r, d] = float(sum(e * Decimal(float(V[b, g, l, d]))
                                                for e, l in zip(ex, vis)) / Z)
    return out


@pytest.mark.parametrize("case", [(1, 2, 1, 6, 3, 2, 3, [6]), (2, 4, 2, 5, 2, 3, 2, [5, 1])])
def test_matches_decimal_bruteforce(case):
    B, h_q, h_kv, n_max, d_k, d_v, T, lens = case
    q = _rand(19, (B, h_q, T, d_k))
    K = _rand(20, (B, h_kv, n_max, d_k))
    V = _rand(21, (B, h_kv, n_max, d_v))
    lens = np.array(lens, np.int32)
    got = oracle.decode_multi(q, K, V, lens, 0.7)
    assert np.max(np.abs(got - _brute_multi(q, K, V, lens, 0.7))) <= 1e-13


def test_append_rows_offsets_and_capacity():
    """Row r of each (b, g) lands at row len[b] + r; rows that do not fit
    are dropped, a negative len is left alone, nothing else moves."""
    B, h_kv, n_max, d, T = 3, 2, 6, 3, 4
    K = np.zeros((B, h_kv, n_max, d), np.float32)
    V = np.zeros((B, h_kv, n_max, 2 * d), np.float32)
    kn = np.arange(B * h_kv * T * d, dtype=np.float32).reshape(B, h_kv, T, d) + 1
    vn = -np.arange(B * h_kv * T * 2 * d, dtype=np.float32).reshape(B, h_kv, T, 2 * d) - 1
    lens = np.array([1, 4, -1], np.int32)
    oracle.append_rows(K, V, kn, vn, lens)
    assert lens.tolist() == [5, 6, -1]
    for g in range(h_kv):
        assert np.array_equal(K[0, g, 1:5], kn[0, g])
        assert np.array_equal(K[1, g, 4:6], kn[1, g, :2])
        assert np.array_equal(V[0, g, 1:5], vn[0, g])
        assert not K[0, g, 0].any() and not K[0, g, 5].any() and not K[1, g, :4].any()
    assert not K[2].any() and not V[2].any()
