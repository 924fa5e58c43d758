"""ctypes binding of ``libhbm_probe.so``: a plain streaming read of two device
buffers, used by the benchmark to measure the machine's practical HBM read
ceiling on the very buffers a decode reads.  Not part of the decode.

Raises ImportError if the library is not built.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY_PATH = os.path.join(_PKG, "libhbm_probe.so")


def _load():
    if not os.path.exists(LIBRARY_PATH):
        raise ImportError(f"{LIBRARY_PATH} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIBRARY_PATH)
    lib.hbm_probe_threads.restype = ctypes.c_int
    lib.hbm_probe_threads.argtypes = []
    lib.hbm_read_probe.restype = ctypes.c_int
    lib.hbm_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                   ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                   ctypes.c_void_p]
    return lib


_lib = _load()
THREADS = _lib.hbm_probe_threads()


def read(a: torch.Tensor, b: torch.Tensor, grid: int = 256, partial=None,
         stream=None) -> torch.Tensor:
    """Stream-read every byte of contiguous device tensors a and b; returns
    (asynchronously) the per-thread sums, grid * THREADS floats."""
    for t in (a, b):
        if not (isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous()):
            raise TypeError("a and b must be contiguous device tensors")
    if partial is None:
        partial = torch.empty(grid * THREADS, dtype=torch.float32, device=a.device)
    s = (stream or torch.cuda.current_stream()).cuda_stream
    st = _lib.hbm_read_probe(a.data_ptr(), a.numel() * a.element_size(), b.data_ptr(),
                             b.numel() * b.element_size(), partial.data_ptr(), int(grid), s)
    if st != 0:
        raise RuntimeError(f"hbm_read_probe failed with status {st}")
    return partial
