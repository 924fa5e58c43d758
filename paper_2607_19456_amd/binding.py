"""Thin ctypes binding of ``libdecode_attn.so`` (the C ABI of
``include/decode_attn.h``) for torch tensors.

Argument marshalling only: every step of the decode runs in the HIP kernels
behind the C ABI.  There is no fallback: if the library is missing or a call
returns an error status, a Python exception is raised.

Tensors must be contiguous, on the current HIP device, float32 (int32 for
``len``).  Calls are asynchronous on torch's current stream (or ``stream``).
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY_PATH = os.environ.get("DECODE_ATTN_LIB", os.path.join(_PKG, "libdecode_attn.so"))

STATUS = {
    0: "DA_OK", 1: "DA_ERR_NULL", 2: "DA_ERR_SHAPE", 3: "DA_ERR_UNSUPPORTED",
    4: "DA_ERR_ALIGN", 5: "DA_ERR_SCALE", 6: "DA_ERR_WORKSPACE", 7: "DA_ERR_HIP",
}

# Every symbol the header declares, with its ctypes signature.
_vp, _ci, _cf, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "da_status_string": (ctypes.c_char_p, [_ci]),
    "da_decode_workspace_bytes": (_sz, [_ci] * 6),
    "da_decode_workspace_counter_bytes": (_sz, [_ci] * 6),
    "da_decode_workspace_reset": (_ci, [_vp, _sz] + [_ci] * 6 + [_vp]),
    "da_decode_attn": (_ci, [_vp, _vp, _vp, _vp, _cf, _vp] + [_ci] * 6 + [_vp, _sz, _vp]),
    "da_decode_step": (_ci, [_vp] * 6 + [_cf, _vp] + [_ci] * 6 + [_vp, _sz, _vp]),
    "da_decode_partial": (_ci, [_vp] * 6 + [_cf] + [_ci] * 6 + [_vp, _sz, _vp]),
    "da_decode_merge": (_ci, [_vp, _vp] + [_ci] * 6 + [_vp, _sz, _vp]),
    "da_decode_multi": (_ci, [_vp, _vp, _vp, _vp, _cf, _vp] + [_ci] * 7 + [_vp, _sz, _vp]),
    "da_decode_multi_step": (_ci, [_vp] * 6 + [_cf, _vp] + [_ci] * 7 + [_vp, _sz, _vp]),
    "da_kv_append": (_ci, [_vp] * 5 + [_ci] * 5 + [_vp]),
    "da_kv_append_rows": (_ci, [_vp] * 5 + [_ci] * 6 + [_vp]),
    "da_decode_attn_noalloc": (_ci, [_vp, _vp, _vp, _vp, _cf, _vp] + [_ci] * 6 + [_vp]),
    # tuning and testing only (explicit segment size)
    "da_decode_chunk_rows": (_ci, [_ci] * 6),
    "da_decode_workspace_bytes_ex": (_sz, [_ci] * 7),
    "da_decode_multi_ex": (_ci, [_vp, _vp, _vp, _vp, _cf, _vp] + [_ci] * 8 + [_vp, _sz, _vp]),
    "da_decode_partial_ex": (_ci, [_vp] * 6 + [_cf] + [_ci] * 8 + [_vp, _sz, _vp]),
    "da_decode_merge_ex": (_ci, [_vp, _vp] + [_ci] * 8 + [_vp, _sz, _vp]),
}


class DecodeAttnError(RuntimeError):
    """A non-OK status from the library."""

    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {_lib.da_status_string(status).decode()}")


def _load():
    if not os.path.exists(LIBRARY_PATH):
        raise ImportError(
            f"HIP library {LIBRARY_PATH} is not built; run __graft_entry__.build() "
            "(there is no CPU fallback)")
    lib = ctypes.CDLL(LIBRARY_PATH)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise DecodeAttnError(fn, status)


def _dev(t: torch.Tensor, name: str, dtype) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise TypeError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def chunk_rows(B, h_q, h_kv, n_max, d_k, d_v) -> int:
    """Segment rows the library picks for these shapes (0: invalid); tuning only."""
    return int(_lib.da_decode_chunk_rows(B, h_q, h_kv, n_max, d_k, d_v))


def workspace_bytes(B, h_q, h_kv, n_max, d_k, d_v, chunk_rows: int = 0) -> int:
    """Workspace bytes a decode with these shapes needs (``chunk_rows`` != 0:
    for the tuning calls with that segment size)."""
    if chunk_rows:
        return int(_lib.da_decode_workspace_bytes_ex(B, h_q, h_kv, n_max, d_k, d_v,
                                                     chunk_rows))
    return int(_lib.da_decode_workspace_bytes(B, h_q, h_kv, n_max, d_k, d_v))


def workspace_counter_bytes(B, h_q, h_kv, n_max, d_k, d_v) -> int:
    """Leading workspace bytes that must be zero before first use."""
    return int(_lib.da_decode_workspace_counter_bytes(B, h_q, h_kv, n_max, d_k, d_v))


def workspace_reset(workspace, B, h_q, h_kv, n_max, d_k, d_v, stream=None) -> None:
    """Zero the counter region of ``workspace`` (h_q counts query rows, h_q*T
    for the T-row calls) with a kernel on the stream."""
    wp, wn = _ws(workspace)
    _check("da_decode_workspace_reset", _lib.da_decode_workspace_reset(
        wp, wn, B, h_q, h_kv, n_max, d_k, d_v, _stream(stream)))


def _shapes(q, K, V):
    if q.dim() != 3 or K.dim() != 4 or V.dim() != 4:
        raise ValueError("q must be [B,h_q,d_k], K [B,h_kv,n_max,d_k], V [B,h_kv,n_max,d_v]")
    B, h_q, d_k = q.shape
    Bk, h_kv, n_max, d_k2 = K.shape
    Bv, h_kv2, n_max2, d_v = V.shape
    if not (B == Bk == Bv and h_kv == h_kv2 and n_max == n_max2 and d_k == d_k2):
        raise ValueError("inconsistent q/K/V shapes")
    return B, h_q, h_kv, n_max, d_k, d_v


def alloc_workspace(q, K, V, chunk_rows: int = 0) -> torch.Tensor:
    """A zeroed workspace for decodes of these shapes (reusable across calls:
    every completed decode leaves its counter region zero again)."""
    B, h_q, h_kv, n_max, d_k, d_v = _shapes(q, K, V)
    n = workspace_bytes(B, h_q, h_kv, n_max, d_k, d_v, chunk_rows)
    if n == 0:
        _check("da_decode_workspace_bytes", 2)
    return torch.zeros(n, dtype=torch.uint8, device=q.device)


def _ws(ws):
    if ws.dtype != torch.uint8 or not ws.is_cuda or not ws.is_contiguous():
        raise TypeError("workspace must be a contiguous uint8 GPU tensor")
    return ws.data_ptr(), ws.numel()


def decode_attn(q, K, V, lens, scale: float, out=None, workspace=None,
                chunk_rows: int = 0, stream=None) -> torch.Tensor:
    """out[b,h,:] = softmax(scale * K[b,g] q[b,h]) V[b,g] over len[b] rows
    (``chunk_rows`` != 0: the tuning call with that segment size)."""
    B, h_q, h_kv, n_max, d_k, d_v = _shapes(q, K, V)
    if out is None:
        out = torch.empty((B, h_q, d_v), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_workspace(q, K, V, chunk_rows)
    wp, wn = _ws(workspace)
    args = (_dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
            _dev(V, "V", torch.float32), _dev(lens, "len", torch.int32),
            float(scale), _dev(out, "out", torch.float32), B, h_q, h_kv, n_max, d_k, d_v)
    if chunk_rows:
        _check("da_decode_multi_ex", _lib.da_decode_multi_ex(
            *args, 1, int(chunk_rows), wp, wn, _stream(stream)))
    else:
        _check("da_decode_attn", _lib.da_decode_attn(*args, wp, wn, _stream(stream)))
    return out


NOALLOC_MAX_WORKSPACE_BYTES = 64 << 20


def decode_attn_noalloc(q, K, V, lens, scale: float, out, stream=None) -> torch.Tensor:
    """decode_attn on the library's own static workspace (no allocation by
    the library; ``out`` is the caller's).  Calls on one GPU must not
    overlap in time."""
    B, h_q, h_kv, n_max, d_k, d_v = _shapes(q, K, V)
    _check("da_decode_attn_noalloc", _lib.da_decode_attn_noalloc(
        _dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
        _dev(V, "V", torch.float32), _dev(lens, "len", torch.int32),
        float(scale), _dev(out, "out", torch.float32), B, h_q, h_kv, n_max, d_k, d_v,
        _stream(stream)))
    return out


def decode_step(q, K, V, k_new, v_new, lens, scale: float, out=None, workspace=None,
                chunk_rows: int = 0, stream=None) -> torch.Tensor:
    """kv_append(K, V, k_new, v_new, lens) then decode_attn(q, K, V, lens),
    fused into two kernel launches, or one where every slab is a single
    segment with h_q / h_kv <= 16 and d_k + d_v <= 256 (``chunk_rows`` != 0:
    always two, through the tuning calls)."""
    B, h_q, h_kv, n_max, d_k, d_v = _shapes(q, K, V)
    _new_rows(k_new, v_new, B, h_kv, d_k, d_v)
    if out is None:
        out = torch.empty((B, h_q, d_v), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_workspace(q, K, V, chunk_rows)
    if chunk_rows:
        decode_partial(q, K, V, lens, scale, workspace, chunk_rows, k_new, v_new, stream)
        return decode_merge(out, workspace, B, h_q, h_kv, n_max, d_k, d_v, chunk_rows,
                            lens, stream)
    wp, wn = _ws(workspace)
    _check("da_decode_step", _lib.da_decode_step(
        _dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
        _dev(V, "V", torch.float32), _dev(k_new, "k_new", torch.float32),
        _dev(v_new, "v_new", torch.float32), _dev(lens, "len", torch.int32),
        float(scale), _dev(out, "out", torch.float32), B, h_q, h_kv, n_max, d_k,
        d_v, wp, wn, _stream(stream)))
    return out


def _new_rows(k_new, v_new, B, h_kv, d_k, d_v):
    if tuple(k_new.shape) != (B, h_kv, d_k) or tuple(v_new.shape) != (B, h_kv, d_v):
        raise ValueError("k_new must be [B,h_kv,d_k] and v_new [B,h_kv,d_v]")


def decode_partial(q, K, V, lens, scale: float, workspace, chunk_rows: int = 0,
                   k_new=None, v_new=None, stream=None, T: int = 1) -> None:
    """Partials of the decode into ``workspace`` (follow with decode_merge).
    With ``k_new``/``v_new`` the partial also performs the fused append.
    ``T`` > 1 or ``chunk_rows`` != 0 go through the tuning call
    (q [B,h_q,T,d_k], k_new/v_new [B,h_kv,T,d] then)."""
    if T == 1 and q.dim() == 3:
        B, h_q, h_kv, n_max, d_k, d_v = _shapes(q, K, V)
    else:
        B, h_q, h_kv, n_max, d_k, d_v, T = _multi_shapes(q, K, V)
    wp, wn = _ws(workspace)
    kp = vp = None
    if k_new is not None or v_new is not None:
        if T == 1 and k_new.dim() == 3:
            _new_rows(k_new, v_new, B, h_kv, d_k, d_v)
        elif (tuple(k_new.shape) != (B, h_kv, T, d_k)
              or tuple(v_new.shape) != (B, h_kv, T, d_v)):
            raise ValueError("k_new must be [B,h_kv,T,d_k] and v_new [B,h_kv,T,d_v]")
        kp = _dev(k_new, "k_new", torch.float32)
        vp = _dev(v_new, "v_new", torch.float32)
    args = (_dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
            _dev(V, "V", torch.float32), kp, vp, _dev(lens, "len", torch.int32),
            float(scale), B, h_q, h_kv, n_max, d_k, d_v)
    if T != 1 or chunk_rows:
        _check("da_decode_partial_ex", _lib.da_decode_partial_ex(
            *args, int(T), int(chunk_rows), wp, wn, _stream(stream)))
    else:
        _check("da_decode_partial", _lib.da_decode_partial(*args, wp, wn, _stream(stream)))


def decode_merge(out, workspace, B, h_q, h_kv, n_max, d_k, d_v,
                 chunk_rows: int = 0, lens=None, stream=None, T: int = 1) -> torch.Tensor:
    """Combine the partials in ``workspace`` into ``out`` (re-zeroes the
    workspace counters).  ``lens``: after a partial with a fused append, the
    lengths to advance.  ``T`` and ``chunk_rows``: those of the partial."""
    wp, wn = _ws(workspace)
    lp = None if lens is None else _dev(lens, "len", torch.int32)
    op = _dev(out, "out", torch.float32)
    if T != 1 or chunk_rows:
        _check("da_decode_merge_ex", _lib.da_decode_merge_ex(
            op, lp, B, h_q, h_kv, n_max, d_k, d_v, int(T), int(chunk_rows), wp, wn,
            _stream(stream)))
    else:
        _check("da_decode_merge", _lib.da_decode_merge(
            op, lp, B, h_q, h_kv, n_max, d_k, d_v, wp, wn, _stream(stream)))
    return out


def kv_append(K, V, k_new, v_new, lens, stream=None) -> None:
    """Write k_new/v_new at row len[b] of every KV head, then len[b] += 1."""
    if K.dim() != 4 or V.dim() != 4:
        raise ValueError("K and V must be [B,h_kv,n_max,d]")
    B, h_kv, n_max, d_k = K.shape
    d_v = V.shape[3]
    if tuple(V.shape[:3]) != (B, h_kv, n_max):
        raise ValueError("K and V disagree in [B,h_kv,n_max]")
    _new_rows(k_new, v_new, B, h_kv, d_k, d_v)
    _check("da_kv_append", _lib.da_kv_append(
        _dev(K, "K", torch.float32), _dev(V, "V", torch.float32),
        _dev(k_new, "k_new", torch.float32), _dev(v_new, "v_new", torch.float32),
        _dev(lens, "len", torch.int32), B, h_kv, n_max, d_k, d_v, _stream(stream)))


# --- several query rows per head (causal) -------------------------------------

def _multi_shapes(q, K, V):
    if q.dim() != 4 or K.dim() != 4 or V.dim() != 4:
        raise ValueError("q must be [B,h_q,T,d_k], K [B,h_kv,n_max,d_k], V [B,h_kv,n_max,d_v]")
    B, h_q, T, d_k = q.shape
    Bk, h_kv, n_max, d_k2 = K.shape
    Bv, h_kv2, n_max2, d_v = V.shape
    if not (B == Bk == Bv and h_kv == h_kv2 and n_max == n_max2 and d_k == d_k2):
        raise ValueError("inconsistent q/K/V shapes")
    return B, h_q, h_kv, n_max, d_k, d_v, T


def alloc_multi_workspace(q, K, V, chunk_rows: int = 0) -> torch.Tensor:
    """A zeroed workspace for multi-row decodes of these shapes (q [B,h_q,T,d_k])."""
    B, h_q, h_kv, n_max, d_k, d_v, T = _multi_shapes(q, K, V)
    n = workspace_bytes(B, h_q * T, h_kv, n_max, d_k, d_v, chunk_rows)
    if n == 0:
        _check("da_decode_workspace_bytes", 2)
    return torch.zeros(n, dtype=torch.uint8, device=q.device)


def decode_multi(q, K, V, lens, scale: float, out=None, workspace=None,
                 chunk_rows: int = 0, stream=None) -> torch.Tensor:
    """T query rows per head, causal: row r of sequence b attends cache rows
    0 .. len[b]-T+r.  q [B,h_q,T,d_k] -> out [B,h_q,T,d_v]."""
    B, h_q, h_kv, n_max, d_k, d_v, T = _multi_shapes(q, K, V)
    if out is None:
        out = torch.empty((B, h_q, T, d_v), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_multi_workspace(q, K, V, chunk_rows)
    wp, wn = _ws(workspace)
    args = (_dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
            _dev(V, "V", torch.float32), _dev(lens, "len", torch.int32),
            float(scale), _dev(out, "out", torch.float32), B, h_q, h_kv, n_max, d_k,
            d_v, T)
    if chunk_rows:
        _check("da_decode_multi_ex", _lib.da_decode_multi_ex(
            *args, int(chunk_rows), wp, wn, _stream(stream)))
    else:
        _check("da_decode_multi", _lib.da_decode_multi(*args, wp, wn, _stream(stream)))
    return out


def decode_multi_step(q, K, V, k_new, v_new, lens, scale: float, out=None,
                      workspace=None, chunk_rows: int = 0, stream=None) -> torch.Tensor:
    """T successive decode steps at once: append k_new/v_new [B,h_kv,T,d] at
    len[b].., then query row r attends rows 0 .. len[b]+r (len on entry)."""
    B, h_q, h_kv, n_max, d_k, d_v, T = _multi_shapes(q, K, V)
    if tuple(k_new.shape) != (B, h_kv, T, d_k) or tuple(v_new.shape) != (B, h_kv, T, d_v):
        raise ValueError("k_new must be [B,h_kv,T,d_k] and v_new [B,h_kv,T,d_v]")
    if out is None:
        out = torch.empty((B, h_q, T, d_v), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_multi_workspace(q, K, V, chunk_rows)
    if chunk_rows:
        decode_partial(q, K, V, lens, scale, workspace, chunk_rows, k_new, v_new, stream, T)
        return decode_merge(out, workspace, B, h_q, h_kv, n_max, d_k, d_v, chunk_rows,
                            lens, stream, T)
    wp, wn = _ws(workspace)
    _check("da_decode_multi_step", _lib.da_decode_multi_step(
        _dev(q, "q", torch.float32), _dev(K, "K", torch.float32),
        _dev(V, "V", torch.float32), _dev(k_new, "k_new", torch.float32),
        _dev(v_new, "v_new", torch.float32), _dev(lens, "len", torch.int32),
        float(scale), _dev(out, "out", torch.float32), B, h_q, h_kv, n_max, d_k,
        d_v, T, wp, wn, _stream(stream)))
    return out


def kv_append_rows(K, V, k_new, v_new, lens, stream=None) -> None:
    """Append T rows per KV head (k_new [B,h_kv,T,d_k]) at len[b].., as many
    as fit; len[b] advances by the rows written."""
    if K.dim() != 4 or V.dim() != 4 or k_new.dim() != 4:
        raise ValueError("K, V must be [B,h_kv,n_max,d] and k_new/v_new [B,h_kv,T,d]")
    B, h_kv, n_max, d_k = K.shape
    d_v = V.shape[3]
    T = k_new.shape[2]
    if tuple(k_new.shape) != (B, h_kv, T, d_k) or tuple(v_new.shape) != (B, h_kv, T, d_v):
        raise ValueError("k_new must be [B,h_kv,T,d_k] and v_new [B,h_kv,T,d_v]")
    _check("da_kv_append_rows", _lib.da_kv_append_rows(
        _dev(K, "K", torch.float32), _dev(V, "V", torch.float32),
        _dev(k_new, "k_new", torch.float32), _dev(v_new, "v_new", torch.float32),
        _dev(lens, "len", torch.int32), B, h_kv, n_max, d_k, d_v, T, _stream(stream)))
