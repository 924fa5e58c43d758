"""Algorithmic byte counts of decode attention and the KV append.

These are the paper's traffic formulas (fp32, 4 bytes per element); the
benchmark divides them by measured kernel time to get achieved bandwidth.
Nothing here touches data.

* Proposition 1 (decode memory minimality), one query head over n rows:
  ``(d_k + n*d_k + n*d_v + d_v) * 4``.
* Proposition 2 (cache-append traffic): ``(d_k + d_v) * 4`` per step,
  independent of the cache length.
* Eq. (8), per-step cost, and Table 4's accounting over T steps:
  append ``T*(d_k+d_v)*4``, decode ``sum_{t=1..T} (d_k + t*d_k + t*d_v + d_v)*4``,
  score matrix ``sum_{t=1..T} t^2 * 4``.
* Table 6 (GQA/MQA): KV read once per KV head ``h_kv*n*(d_k+d_v)*4``; the
  total adds one query read and one output write per query head,
  ``h_q*(d_k+d_v)*4``.
* Table 2's comparison column: the n x n score matrix, ``n^2 * 4``.
"""
from __future__ import annotations

from typing import Iterable

F32 = 4


def decode_bytes(n: int, d_k: int, d_v: int) -> int:
    """Proposition 1: bytes one single-query decode over n rows must move."""
    return (d_k + n * d_k + n * d_v + d_v) * F32


def score_matrix_bytes(n: int) -> int:
    """Table 2: bytes of the n x n score matrix the standard formula forms."""
    return n * n * F32


def append_bytes(d_k: int, d_v: int) -> int:
    """Proposition 2: bytes one KV append writes (one K row, one V row)."""
    return (d_k + d_v) * F32


def step_bytes(t: int, d_k: int, d_v: int) -> int:
    """Eq. (8): the append plus the decode's K and V rows over t cached
    rows (eq. (8) leaves out Proposition 1's query and output terms)."""
    return append_bytes(d_k, d_v) + (t * d_k + t * d_v) * F32


def multistep_table(T: int, d_k: int, d_v: int) -> tuple[int, int, int]:
    """Table 4: (append, decode, score-matrix) bytes summed over T steps."""
    app = T * append_bytes(d_k, d_v)
    dec = sum(decode_bytes(t, d_k, d_v) for t in range(1, T + 1))
    n2 = sum(t * t * F32 for t in range(1, T + 1))
    return app, dec, n2


def gqa_table(n: int, d_k: int, d_v: int, h_q: int, h_kv: int) -> tuple[int, int]:
    """Table 6: (KV, total) bytes of one GQA/MQA decode step."""
    kv = h_kv * n * (d_k + d_v) * F32
    return kv, kv + h_q * (d_k + d_v) * F32


def batch_decode_bytes(lens: Iterable[int], h_q: int, h_kv: int, d_k: int,
                       d_v: int, rows: int = 1) -> int:
    """Decode over a batch: every KV head of sequence b read once over its
    len_b rows (Table 6's KV term), plus each query head's q read and output
    write (Table 6's total), for each of ``rows`` query rows per head."""
    lens = [max(0, int(n)) for n in lens]
    kv = sum(h_kv * n * (d_k + d_v) * F32 for n in lens)
    return kv + len(lens) * h_q * rows * (d_k + d_v) * F32


def batch_partial_bytes(lens: Iterable[int], h_q: int, h_kv: int, d_k: int,
                        d_v: int, rows: int = 1) -> int:
    """Bytes the split-partial kernel must read: K and V over the valid rows
    of every KV head, and every query vector (the output row is written by
    the merge)."""
    lens = [max(0, int(n)) for n in lens]
    kv = sum(h_kv * n * (d_k + d_v) * F32 for n in lens)
    return kv + len(lens) * h_q * rows * d_k * F32


def batch_append_bytes(B: int, h_kv: int, d_k: int, d_v: int, rows: int = 1) -> int:
    """Proposition 2 over a batch: one K row and one V row per KV head (per
    appended position)."""
    return B * h_kv * rows * append_bytes(d_k, d_v)
