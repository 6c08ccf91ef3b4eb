"""On-Demand Attention (ODA) decode-step hot path for AMD MI355X (gfx950).

The product is the C-ABI library ``liboda.so`` (include/oda.h): hand-written
HIP kernels for Local decode attention (over the paged cache, or over the
direct-ring workspace), the recall gate with its device predicate, Full
decode attention for flagged requests only, the selected-state commit, and
the decoder layers around them (``decoder`` composes a whole
synthetic decode step from those entry points).  This package
holds its sources (``csrc/``), its build step (``build.py``), a ctypes
binding with the same entry-point names (``_lib``), the byte accounting used
to report bandwidth (``ledger``) and the synthetic workload shapes
(``workloads``).

The binding is loaded on first use of any entry point; if ``liboda.so`` has
not been built that raises ImportError (there is no fallback path).
"""
_EXPORTS = ("HEAD_MLP", "HEAD_PAPER", "OdaError", "Shape", "attn_workspace_size", "full_decode_attn",
            "gate_desc", "gate_param_count", "gate_workspace_size", "inputs", "local_decode_attn",
            "recall_gate", "lib", "prepare_local", "prepare_full", "prepare_gate", "Call", "commit_kv", "prepare_commit",
            "commit_workspace_size",
            "DENSE_PLAIN", "DENSE_SWIGLU", "dense_desc", "dense_bf16", "qk_norm_rope", "embed_bf16", "copy_rows",
            "argmax", "prepare_dense", "prepare_qk_norm_rope", "prepare_embed", "prepare_copy_rows",
            "prepare_argmax", "stream_read", "prepare_stream_read", "rms_norm_rows", "prepare_rms_norm_rows",
            "recall_gate_static", "qkv_prep", "prepare_local_qkv", "prepare_full_qkv",
            "ring_elements", "ring_fill", "local_decode_attn_ring", "commit_kv_ring", "prepare_local_ring")


def __getattr__(name):
    if name in _EXPORTS:
        from . import _lib
        return _lib if name == "lib" else getattr(_lib, name)
    raise AttributeError(name)
