"""Seeded synthetic workloads for decode attention.

This module only draws random numbers and fixes shapes: it holds none of the
method's arithmetic.  Both the HIP path (through the tests and the benchmark)
and the CPU oracle consume the very same bytes it produces.

Inputs are i.i.d. N(0, 1) fp32, as in the paper's experiments (synthetic
float32 tensors from a fixed seed; the paper fixes no generator).  Normals
come from ``csrc/workload_rng.c``: Philox4x32-10 counters (seed, stream,
index) turned into normals by Box-Muller, so element i of a stream is the
same for any thread count and any machine with IEEE doubles and a correctly
behaved libm.

Draw order (each item its own stream id): initial lengths, q, K, V, then for
every step s: k_new[s], v_new[s], q[s].  Cache rows at or beyond a
sequence's length are filled with ``pad`` (NaN in parity tests so that a
kernel that reads them is caught, 0 in the benchmark).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "workload_rng.c")
_LIB = os.path.join(_HERE, "libworkload_rng.so")
_lib = None


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover - non-Linux
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def build_rng(force: bool = False) -> str:
    """Compile the generator with gcc (plain C, OpenMP).  Returns its path."""
    if force or not os.path.exists(_LIB) or (
            os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                        "-fopenmp", "-fno-fast-math", "-Wall", "-o", tmp, _SRC,
                        "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _rng():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build_rng())
        lib.workload_normal_f32.argtypes = [
            ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
            ctypes.POINTER(ctypes.c_float), ctypes.c_int64, ctypes.c_int]
        lib.workload_normal_f32.restype = None
        u32p = ctypes.POINTER(ctypes.c_uint32)
        lib.workload_philox4x32_10.argtypes = [u32p, u32p, u32p]
        lib.workload_philox4x32_10.restype = None
        _lib = lib
    return _lib


def philox4x32_10(ctr, key) -> list:
    """One Philox4x32-10 block (exposed for the published test vectors)."""
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    _rng().workload_philox4x32_10(c, k, o)
    return list(o)


def fill_normal(out: np.ndarray, seed: int, stream: int, offset: int = 0,
                threads: int | None = None) -> None:
    """Fill the contiguous float32 array ``out`` with samples
    ``offset .. offset + out.size`` of stream (seed, stream)."""
    assert out.dtype == np.float32 and out.flags.c_contiguous
    if out.size:
        _rng().workload_normal_f32(
            int(seed), int(stream), int(offset),
            out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), int(out.size),
            int(threads or _threads()))


def normal(seed: int, stream: int, shape, threads: int | None = None) -> np.ndarray:
    """float32 N(0,1) array of ``shape``; identical for any thread count."""
    out = np.empty(shape, dtype=np.float32)
    fill_normal(out, seed, stream, 0, threads)
    return out


def cache(seed: int, stream: int, lens: np.ndarray, h_kv: int, n_max: int,
          d: int, pad: float, threads: int | None = None) -> np.ndarray:
    """A [B, h_kv, n_max, d] cache whose valid rows hold the samples of the
    flat array ``normal(seed, stream, (B, h_kv, n_max, d))`` and whose rows at
    or beyond ``lens[b]`` hold ``pad``.  Only valid rows are drawn."""
    B = int(lens.shape[0])
    out = np.empty((B, h_kv, n_max, d), dtype=np.float32)
    for b in range(B):
        n = min(max(0, int(lens[b])), n_max)
        for g in range(h_kv):
            slab = out[b, g]
            base = ((b * h_kv + g) * n_max) * d
            if n:
                fill_normal(slab[:n].reshape(-1), seed, stream, base, threads)
            slab[n:] = pad
    return out


@dataclass(frozen=True)
class Shape:
    """Shapes of one decode-attention workload.

    ``len_lo``/``len_hi`` bound the initial per-sequence lengths (inclusive);
    ``steps`` is the number of (append, decode) steps (0: one decode of the
    initial cache, no append); ``rows`` is the number of positions a step
    submits at once (query rows per head and rows appended per KV head;
    1: the single-query decode)."""
    name: str
    B: int
    h_q: int
    h_kv: int
    d_k: int
    d_v: int
    n_max: int
    len_lo: int
    len_hi: int
    steps: int
    scale: float = field(default=0.0)
    description: str = ""
    rows: int = 1

    @property
    def G(self) -> int:
        return self.h_q // self.h_kv

    def scale32(self) -> np.float32:
        s = self.scale if self.scale else 1.0 / math.sqrt(self.d_k)
        return np.float32(s)


# The five workloads the path is measured and checked on.
WORKLOADS = {
    "mha1_d64_n128": Shape(
        "mha1_d64_n128", B=1, h_q=1, h_kv=1, d_k=64, d_v=64, n_max=128,
        len_lo=128, len_hi=128, steps=0,
        description="single decode step, one MHA head, d=64, n=128"),
    "mha32_b8_d128_n4096_16steps": Shape(
        "mha32_b8_d128_n4096_16steps", B=8, h_q=32, h_kv=32, d_k=128, d_v=128,
        n_max=4112, len_lo=4096, len_hi=4096, steps=16,
        description="MHA decode, B=8, 32 heads, d=128, n=4096, 16 append+decode steps"),
    "gqa32x8_b16_d128_n8192": Shape(
        "gqa32x8_b16_d128_n8192", B=16, h_q=32, h_kv=8, d_k=128, d_v=128,
        n_max=8192, len_lo=8192, len_hi=8192, steps=0,
        description="GQA decode (group 4), B=16, d=128, n=8192, one step"),
    "mqa32_b32_d128_n16384": Shape(
        "mqa32_b32_d128_n16384", B=32, h_q=32, h_kv=1, d_k=128, d_v=128,
        n_max=16384, len_lo=16384, len_hi=16384, steps=0,
        description="MQA decode, B=32, 32 query heads, d=128, n=16384, one step"),
    "gqa64x8_b4_d128_ragged64k-128k_64steps": Shape(
        "gqa64x8_b4_d128_ragged64k-128k_64steps", B=4, h_q=64, h_kv=8, d_k=128,
        d_v=128, n_max=131072, len_lo=65536, len_hi=131072 - 64, steps=64,
        description="long-context ragged GQA (group 8), B=4, d=128, "
                    "len ~ U{65536..131008}, n_max=131072, 64 append+decode steps"),
    # Several positions per step (speculative verification of 4 draft tokens)
    # on the long-context workload: the same 64 positions in 16 steps.
    "gqa64x8_b4_d128_ragged64k-128k_16steps_x4rows": Shape(
        "gqa64x8_b4_d128_ragged64k-128k_16steps_x4rows", B=4, h_q=64, h_kv=8, d_k=128,
        d_v=128, n_max=131072, len_lo=65536, len_hi=131072 - 64, steps=16, rows=4,
        description="long-context ragged GQA (group 8), B=4, d=128, "
                    "len ~ U{65536..131008}, 16 steps of 4 positions each "
                    "(4 rows appended, 4 causal query rows per head)"),
}

# Short aliases used on command lines and in test ids.
ALIASES = {
    "c1": "mha1_d64_n128",
    "c2": "mha32_b8_d128_n4096_16steps",
    "c3": "gqa32x8_b16_d128_n8192",
    "c4": "mqa32_b32_d128_n16384",
    "c5": "gqa64x8_b4_d128_ragged64k-128k_64steps",
    "spec4": "gqa64x8_b4_d128_ragged64k-128k_16steps_x4rows",
}


def get(name: str) -> Shape:
    return WORKLOADS[ALIASES.get(name, name)]


@dataclass
class Inputs:
    shape: Shape
    lens: np.ndarray            # int32 [B], initial lengths
    q: np.ndarray               # float32 [B, h_q, d_k], query of the first decode
                                # ([B, h_q, rows, d_k] when rows > 1)
    K: np.ndarray               # float32 [B, h_kv, n_max, d_k]
    V: np.ndarray               # float32 [B, h_kv, n_max, d_v]
    k_new: np.ndarray           # float32 [steps, B, h_kv, d_k]   (rows > 1: [.., rows, d_k])
    v_new: np.ndarray           # float32 [steps, B, h_kv, d_v]   (rows > 1: [.., rows, d_v])
    q_step: np.ndarray          # float32 [steps, B, h_q, d_k]    (rows > 1: [.., rows, d_k])


def draw_lengths(shape: Shape, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, 0])
    return rng.integers(shape.len_lo, shape.len_hi, size=shape.B,
                        endpoint=True).astype(np.int32)


def make(shape: Shape, seed: int = 0, pad: float = float("nan"),
         lens: np.ndarray | None = None, threads: int | None = None) -> Inputs:
    """Draw a full workload.  ``lens`` overrides the drawn initial lengths."""
    s = shape
    if lens is None:
        lens = draw_lengths(s, seed)
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    r = () if s.rows == 1 else (s.rows,)
    q = normal(seed, 1, (s.B, s.h_q) + r + (s.d_k,), threads)
    K = cache(seed, 2, lens, s.h_kv, s.n_max, s.d_k, pad, threads)
    V = cache(seed, 3, lens, s.h_kv, s.n_max, s.d_v, pad, threads)
    kn = np.empty((s.steps, s.B, s.h_kv) + r + (s.d_k,), np.float32)
    vn = np.empty((s.steps, s.B, s.h_kv) + r + (s.d_v,), np.float32)
    qs = np.empty((s.steps, s.B, s.h_q) + r + (s.d_k,), np.float32)
    for t in range(s.steps):
        kn[t] = normal(seed, 4 + 3 * t, kn.shape[1:], threads)
        vn[t] = normal(seed, 5 + 3 * t, vn.shape[1:], threads)
        qs[t] = normal(seed, 6 + 3 * t, qs.shape[1:], threads)
    return Inputs(s, lens, q, K, V, kn, vn, qs)


def custom(name: str = "custom", *, B: int, h_q: int, h_kv: int, d_k: int,
           d_v: int, n_max: int, len_lo: int | None = None,
           len_hi: int | None = None, steps: int = 0,
           scale: float = 0.0, rows: int = 1) -> Shape:
    """A workload of arbitrary shape (tests: ragged tails, edge cases)."""
    lo = n_max if len_lo is None else len_lo
    hi = lo if len_hi is None else len_hi
    return Shape(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v, n_max=n_max,
                 len_lo=lo, len_hi=hi, steps=steps, scale=scale, rows=rows)
