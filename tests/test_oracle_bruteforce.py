"""The oracle against a high-precision brute force on tiny inputs.

The brute force takes another route to the same definition: Python
``decimal`` at 50 significant digits, the textbook softmax without the max
subtraction, and the GQA head map by explicitly repeating each KV head
G = h_q/h_kv times (the standard expansion the GQA section compares against)
instead of computing the KV head index.
"""
from decimal import Decimal, getcontext

import numpy as np
import pytest

import oracle

getcontext().prec = 50


def _brute(q, K, V, lens, scale):
    B, h_q, d_k = q.shape
    _, h_kv, n_max, _ = K.shape
    d_v = V.shape[3]
    G = h_q // h_kv
    Kx = np.repeat(K, G, axis=1)   # [B, h_q, n_max, d_k]
    Vx = np.repeat(V, G, axis=1)
    sc = Decimal(float(np.float32(scale)))
    out = np.zeros((B, h_q, d_v))
    for b in range(B):
        n = min(max(int(lens[b]), 0), n_max)
        for h in range(h_q):
            if n == 0:
                continue
            ex = []
            for l in range(n):
                dot = sum(Decimal(float(q[b, h, j])) * Decimal(float(Kx[b, h, l, j]))
                          for j in range(d_k))
                ex.append((sc * dot).exp())
            Z = sum(ex)
            for d in range(d_v):
                num = sum(ex[l] * Decimal(float(Vx[b, h, l, d])) for l in range(n))
                out[b, h, d] = float(num / Z)
    return out


CASES = [
    # B, h_q, h_kv, n_max, d_k, d_v, lens
    (1, 1, 1, 1, 1, 1, [1]),
    (1, 1, 1, 5, 3, 2, [5]),
    (2, 4, 2, 6, 4, 3, [6, 3]),
    (2, 4, 1, 7, 2, 4, [7, 1]),
    (1, 3, 3, 8, 4, 4, [5]),
    (2, 2, 2, 4, 3, 5, [0, 4]),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("seed", [0, 1])
def test_oracle_matches_decimal_bruteforce(case, seed):
    B, h_q, h_kv, n_max, d_k, d_v, lens = case
    rng = np.random.default_rng([seed, B, h_q, h_kv, n_max])
    q = rng.standard_normal((B, h_q, d_k)).astype(np.float32)
    K = (2 * rng.standard_normal((B, h_kv, n_max, d_k))).astype(np.float32)
    V = rng.standard_normal((B, h_kv, n_max, d_v)).astype(np.float32)
    lens = np.array(lens, np.int32)
    scale = np.float32(0.9)
    got = oracle.decode(q, K, V, lens, scale)
    ref = _brute(q, K, V, lens, scale)
    assert np.max(np.abs(got - ref)) <= 1e-13


def test_bruteforce_catches_large_logits():
    """Scores up to ~80: the brute force needs no max subtraction, the
    oracle does (fp64 exp of 80 is fine too, but the weights span e^-160)."""
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 2, 4)).astype(np.float32) * 4
    K = rng.standard_normal((1, 1, 6, 4)).astype(np.float32) * 4
    V = rng.standard_normal((1, 1, 6, 3)).astype(np.float32)
    lens = np.array([6], np.int32)
    got = oracle.decode(q, K, V, lens, np.float32(1.0))
    ref = _brute(q, K, V, lens, np.float32(1.0))
    assert np.max(np.abs(got - ref)) <= 1e-13
