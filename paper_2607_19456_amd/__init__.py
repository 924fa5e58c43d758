"""MI355X (gfx950) decode attention over a KV cache: MHA/GQA/MQA decode and
the per-step KV append, after "MoA-Structured Decode Attention" (Mullin and
Hains, 2026).

The compute lives in the HIP library ``libdecode_attn.so`` behind the C ABI
of ``include/decode_attn.h``; :mod:`.binding` marshals torch tensors into it.
The binding is imported on first use of one of its names, so the workload
generator and the traffic model stay importable on machines without the
built library; using the decode or append without it raises ImportError.
"""
from importlib import import_module

_BINDING_NAMES = {
    "decode_attn", "decode_attn_noalloc", "decode_step", "decode_partial", "decode_merge", "kv_append",
    "decode_multi", "decode_multi_step", "kv_append_rows", "alloc_multi_workspace",
    "chunk_rows", "workspace_bytes", "workspace_counter_bytes", "workspace_reset",
    "alloc_workspace", "DecodeAttnError",
    "LIBRARY_PATH",
}

__all__ = sorted(_BINDING_NAMES)


def __getattr__(name):
    if name in _BINDING_NAMES:
        return getattr(import_module(".binding", __name__), name)
    raise AttributeError(name)
