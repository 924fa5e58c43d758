"""CPU oracle for single-query decode attention and the KV append.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the benchmark's ``cpu_baseline`` leg may import this package.  The
product path (``paper_2607_19456_amd``) never imports, links or calls it, and
the two share no code: the oracle's arithmetic lives in ``oracle.c`` (plain
fp64 loops following Algorithm 1 of the paper), this module only marshals
numpy arrays into it.

Functions follow the paper as follows:

* :func:`decode` -- Algorithm 1 (eqs. (1)-(3)) lifted over batch and query
  heads, with the psi-selection head map of eq. (10) for GQA/MQA.
* :func:`decode_weights` -- Step II's weight vector for one (b, h).
* :func:`append` -- the concatenation append of eqs. (6)-(7) with the
  semantics of the multi-step section's pre-allocated cache.
* :func:`decode_multi` -- T query rows per head with causal visibility (the
  rank-2 query of the paper's training form, for a step that submits several
  positions at once): each row is Algorithm 1 on its causal prefix.
* :func:`append_rows` -- :func:`append` applied T times in order.

Every function is pinned by ``tests/test_oracle_*.py`` against the paper's
worked examples, closed forms, invariants, a high-precision brute force and
PyTorch's SDPA (the paper's own ground truth).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc (-O2, no fast-math,
    OpenMP over the independent (b, h) units).  Returns the library path."""
    if force or not os.path.exists(_LIB) or (
            os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    return _configure(ctypes.CDLL(_LIB))


def _configure(lib):
    global _lib
    f32p = ctypes.POINTER(ctypes.c_float)
    f64p = ctypes.POINTER(ctypes.c_double)
    i32p = ctypes.POINTER(ctypes.c_int32)
    u8p = ctypes.POINTER(ctypes.c_uint8)
    ci = ctypes.c_int
    lib.oracle_decode.argtypes = [f32p, f32p, f32p, i32p, ctypes.c_float,
                                  f64p, ci, ci, ci, ci, ci, ci, u8p, ci]
    lib.oracle_decode.restype = ci
    lib.oracle_decode_weights.argtypes = [f32p, f32p, f32p, i32p,
                                          ctypes.c_float, ci, ci, ci, ci, ci,
                                          ci, ci, ci, f64p, f64p]
    lib.oracle_decode_weights.restype = ctypes.c_int64
    lib.oracle_append.argtypes = [f32p, f32p, f32p, f32p, i32p,
                                  ci, ci, ci, ci, ci]
    lib.oracle_append.restype = ci
    lib.oracle_decode_multi.argtypes = [f32p, f32p, f32p, i32p, ctypes.c_float,
                                        f64p, ci, ci, ci, ci, ci, ci, ci, ci]
    lib.oracle_decode_multi.restype = ci
    lib.oracle_append_rows.argtypes = [f32p, f32p, f32p, f32p, i32p,
                                       ci, ci, ci, ci, ci, ci]
    lib.oracle_append_rows.restype = ci
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ci
    _lib = lib
    return lib


class use_library:
    """Context manager: route this module's calls to another build of the
    oracle (used only by the mutation test, which plants mistakes in copies
    of ``oracle.c`` to show that the pins catch them)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self._saved = _lib
        _lib = None
        _configure(ctypes.CDLL(self.path))
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self._saved
        return False


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f32(a, name, ndim):
    if not (isinstance(a, np.ndarray) and a.dtype == np.float32
            and a.flags.c_contiguous and a.ndim == ndim):
        raise TypeError(f"{name}: need a C-contiguous float32 array of rank {ndim}")
    return a


def _lens(a, B):
    a = np.ascontiguousarray(a, dtype=np.int32)
    if a.shape != (B,):
        raise ValueError(f"len: need shape ({B},), got {a.shape}")
    return a


def max_threads() -> int:
    """OpenMP threads the oracle uses by default (OMP_NUM_THREADS honoured)."""
    return int(_load().oracle_max_threads())


def decode(q, K, V, lens, scale, heads=None, threads: int = 0) -> np.ndarray:
    """Decode attention for every (b, h): returns ``out[B, h_q, d_v]`` (fp64).

    q[B,h_q,d_k], K[B,h_kv,n_max,d_k], V[B,h_kv,n_max,d_v] float32, lens[B]
    int32, scale a float32 value.  ``heads`` optionally restricts the work to
    a boolean mask of shape (B, h_q); rows of masked-out heads are NaN.
    """
    lib = _load()
    q = _f32(q, "q", 3)
    K = _f32(K, "K", 4)
    V = _f32(V, "V", 4)
    B, h_q, d_k = q.shape
    Bk, h_kv, n_max, d_k2 = K.shape
    Bv, h_kv2, n_max2, d_v = V.shape
    if not (Bk == Bv == B and h_kv2 == h_kv and n_max2 == n_max and d_k2 == d_k):
        raise ValueError("inconsistent q/K/V shapes")
    lens = _lens(lens, B)
    out = np.full((B, h_q, d_v), np.nan, dtype=np.float64)
    mask_p = None
    if heads is not None:
        heads = np.ascontiguousarray(heads, dtype=np.uint8)
        if heads.shape != (B, h_q):
            raise ValueError("heads mask must have shape (B, h_q)")
        mask_p = _ptr(heads, ctypes.c_uint8)
    rc = lib.oracle_decode(_ptr(q, ctypes.c_float), _ptr(K, ctypes.c_float),
                           _ptr(V, ctypes.c_float), _ptr(lens, ctypes.c_int32),
                           ctypes.c_float(np.float32(scale)),
                           _ptr(out, ctypes.c_double), B, h_q, h_kv, n_max,
                           d_k, d_v, mask_p, int(threads))
    if rc != 0:
        raise ValueError("oracle_decode rejected the shapes (h_kv must divide h_q)")
    return out


def decode_weights(q, K, V, lens, scale, b: int, h: int):
    """Step II weights ``a[0..n)`` and the output row of one (b, h)."""
    lib = _load()
    q = _f32(q, "q", 3)
    K = _f32(K, "K", 4)
    V = _f32(V, "V", 4)
    B, h_q, d_k = q.shape
    _, h_kv, n_max, _ = K.shape
    d_v = V.shape[3]
    lens = _lens(lens, B)
    w = np.zeros(max(n_max, 1), dtype=np.float64)
    row = np.zeros(d_v, dtype=np.float64)
    n = lib.oracle_decode_weights(
        _ptr(q, ctypes.c_float), _ptr(K, ctypes.c_float),
        _ptr(V, ctypes.c_float), _ptr(lens, ctypes.c_int32),
        ctypes.c_float(np.float32(scale)), int(b), int(h), B, h_q, h_kv, n_max,
        d_k, d_v, _ptr(w, ctypes.c_double), _ptr(row, ctypes.c_double))
    if n < 0:
        raise ValueError("oracle_decode_weights rejected its arguments")
    return w[:n].copy(), row


def append(K, V, k_new, v_new, lens) -> None:
    """In-place KV append on host arrays; ``lens`` (int32 ndarray) is updated."""
    lib = _load()
    K = _f32(K, "K", 4)
    V = _f32(V, "V", 4)
    B, h_kv, n_max, d_k = K.shape
    d_v = V.shape[3]
    k_new = _f32(k_new, "k_new", 3)
    v_new = _f32(v_new, "v_new", 3)
    if k_new.shape != (B, h_kv, d_k) or v_new.shape != (B, h_kv, d_v):
        raise ValueError("k_new/v_new shapes do not match the cache")
    if not (isinstance(lens, np.ndarray) and lens.dtype == np.int32
            and lens.shape == (B,) and lens.flags.c_contiguous):
        raise TypeError("lens must be a contiguous int32 array of shape (B,)")
    rc = lib.oracle_append(_ptr(K, ctypes.c_float), _ptr(V, ctypes.c_float),
                           _ptr(k_new, ctypes.c_float), _ptr(v_new, ctypes.c_float),
                           _ptr(lens, ctypes.c_int32), B, h_kv, n_max, d_k, d_v)
    if rc != 0:
        raise ValueError("oracle_append rejected the shapes")


def decode_multi(q, K, V, lens, scale, threads: int = 0) -> np.ndarray:
    """Decode with T query rows per (b, h): returns ``out[B, h_q, T, d_v]``
    (fp64).  q[B,h_q,T,d_k]; row r of sequence b sits at cache position
    clamp(len[b]) - T + r and attends rows 0..that position."""
    lib = _load()
    q = _f32(q, "q", 4)
    K = _f32(K, "K", 4)
    V = _f32(V, "V", 4)
    B, h_q, T, d_k = q.shape
    Bk, h_kv, n_max, d_k2 = K.shape
    Bv, h_kv2, n_max2, d_v = V.shape
    if not (Bk == Bv == B and h_kv2 == h_kv and n_max2 == n_max and d_k2 == d_k):
        raise ValueError("inconsistent q/K/V shapes")
    lens = _lens(lens, B)
    out = np.full((B, h_q, T, d_v), np.nan, dtype=np.float64)
    rc = lib.oracle_decode_multi(_ptr(q, ctypes.c_float), _ptr(K, ctypes.c_float),
                                 _ptr(V, ctypes.c_float), _ptr(lens, ctypes.c_int32),
                                 ctypes.c_float(np.float32(scale)),
                                 _ptr(out, ctypes.c_double), B, h_q, h_kv, n_max,
                                 d_k, d_v, T, int(threads))
    if rc != 0:
        raise ValueError("oracle_decode_multi rejected the shapes")
    return out


def append_rows(K, V, k_new, v_new, lens) -> None:
    """T rows appended in order (k_new[B,h_kv,T,d_k], v_new[B,h_kv,T,d_v]);
    ``lens`` is updated in place."""
    lib = _load()
    K = _f32(K, "K", 4)
    V = _f32(V, "V", 4)
    B, h_kv, n_max, d_k = K.shape
    d_v = V.shape[3]
    k_new = _f32(k_new, "k_new", 4)
    v_new = _f32(v_new, "v_new", 4)
    T = k_new.shape[2]
    if k_new.shape != (B, h_kv, T, d_k) or v_new.shape != (B, h_kv, T, d_v):
        raise ValueError("k_new/v_new shapes do not match the cache")
    if not (isinstance(lens, np.ndarray) and lens.dtype == np.int32
            and lens.shape == (B,) and lens.flags.c_contiguous):
        raise TypeError("lens must be a contiguous int32 array of shape (B,)")
    rc = lib.oracle_append_rows(_ptr(K, ctypes.c_float), _ptr(V, ctypes.c_float),
                                _ptr(k_new, ctypes.c_float), _ptr(v_new, ctypes.c_float),
                                _ptr(lens, ctypes.c_int32), B, h_kv, n_max, d_k, d_v, T)
    if rc != 0:
        raise ValueError("oracle_append_rows rejected the shapes")
