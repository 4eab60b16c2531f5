"""MI355X-native paged KV hot path for multi-turn agent serving.

kv_append, prefix_prefill_attn and paged_decode_attn are thin bindings of
the HIP library libckv.so (C ABI in include/ckv.h).  The library is loaded
on first use of any of them and a missing build raises ImportError; there
is no other implementation to fall back to.
"""
import importlib

_BINDINGS = ("Batch", "CkvError", "Pool", "decode_workspace_bytes", "kv_append", "paged_decode_attn",
             "prefill_workspace_bytes", "prefix_prefill_attn", "status_string", "validate_batch",
             "version")


def __getattr__(name):
    if name in _BINDINGS:
        return getattr(importlib.import_module(".ckv", __name__), name)
    raise AttributeError(name)
