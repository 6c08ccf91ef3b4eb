"""ctypes binding of liboda.so (include/oda.h).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the library.  torch tensors supply device memory and the current
stream.  If the library is not built, importing this module fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liboda.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_20734_amd.build` "
                      "(or __graft_entry__.build()) before using the HIP path")

# torch's wheel carries its own HIP and HSA runtimes.  Importing torch before
# the library makes the dynamic loader resolve the library's libamdhip64
# against torch's copy, so the process holds one runtime.  Loaded first, the
# library would map the system's runtime beside torch's, and whichever of the
# two HSA runtimes starts second finds no GPU ("no ROCm-capable device").
import torch  # noqa: E402,F401  (load order; the tensors come from torch anyway)

_lib = ctypes.CDLL(LIB_PATH)

ODA_OK = 0
ODA_ERR_NULL = -1
ODA_ERR_SHAPE = -2
ODA_ERR_UNSUPPORTED = -3
ODA_ERR_WORKSPACE = -4
ODA_ERR_HIP = -5

HEAD_PAPER = 0
HEAD_MLP = 1

DENSE_PLAIN = 0
DENSE_SWIGLU = 1

EXPORTED = ("oda_attn_workspace_size", "oda_local_decode_attn", "oda_full_decode_attn",
            "oda_local_decode_attn_qkv", "oda_full_decode_attn_qkv",
            "oda_gate_param_count", "oda_gate_workspace_size", "oda_recall_gate", "oda_recall_gate_static",
            "oda_commit_workspace_size", "oda_commit_kv",
            "oda_ring_elements", "oda_ring_fill", "oda_local_decode_attn_ring", "oda_commit_kv_ring",
            "oda_dense_bf16", "oda_qk_norm_rope", "oda_embed_bf16", "oda_copy_rows", "oda_rms_norm_rows",
            "oda_argmax", "oda_stream_read", "oda_status_string", "oda_last_error")


class OdaError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{status_string(status)} ({detail})")
        self.status = status
        self.detail = detail


class AttnShape(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("max_blocks_per_seq", ctypes.c_int32), ("max_seq_len", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64), ("split_blocks", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("layer_stride_kv", ctypes.c_int64)]


class AttnInputs(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p), ("seq_lens", ctypes.c_void_p),
                ("k_cur", ctypes.c_void_p), ("v_cur", ctypes.c_void_p), ("scale", ctypes.c_float)]


class QkvPrep(ctypes.Structure):
    _fields_ = [("qkv", ctypes.c_void_p), ("q_gain", ctypes.c_void_p), ("k_gain", ctypes.c_void_p),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_double), ("k_out", ctypes.c_void_p),
                ("v_out", ctypes.c_void_p)]


class GateDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("d_model", ctypes.c_int32), ("d_hidden", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("params", ctypes.c_void_p)]


class DenseDesc(ctypes.Structure):
    _fields_ = [("in_features", ctypes.c_int32), ("out_features", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("weight", ctypes.c_void_p), ("norm_gain", ctypes.c_void_p)]


_P = ctypes.POINTER
_V = ctypes.c_void_p
_lib.oda_attn_workspace_size.argtypes = [_P(AttnShape), ctypes.c_int32, ctypes.c_int32, _P(ctypes.c_size_t)]
_lib.oda_attn_workspace_size.restype = ctypes.c_int
_lib.oda_local_decode_attn.argtypes = [_P(AttnShape), _P(AttnInputs), ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p]
_lib.oda_local_decode_attn.restype = ctypes.c_int
_lib.oda_full_decode_attn.argtypes = [_P(AttnShape), _P(AttnInputs), ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
_lib.oda_full_decode_attn.restype = ctypes.c_int
_lib.oda_local_decode_attn_qkv.argtypes = [_P(AttnShape), _P(AttnInputs), _P(QkvPrep), ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_size_t, ctypes.c_void_p]
_lib.oda_local_decode_attn_qkv.restype = ctypes.c_int
_lib.oda_full_decode_attn_qkv.argtypes = [_P(AttnShape), _P(AttnInputs), _P(QkvPrep), ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
_lib.oda_full_decode_attn_qkv.restype = ctypes.c_int
_lib.oda_gate_param_count.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P(ctypes.c_int64)]
_lib.oda_gate_param_count.restype = ctypes.c_int
_lib.oda_gate_workspace_size.argtypes = [_P(GateDesc), ctypes.c_int32, _P(ctypes.c_size_t)]
_lib.oda_gate_workspace_size.restype = ctypes.c_int
_lib.oda_recall_gate.argtypes = [_P(GateDesc), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
_lib.oda_recall_gate.restype = ctypes.c_int
_lib.oda_recall_gate_static.argtypes = [_P(GateDesc), ctypes.c_int32, _V, _V, _V, ctypes.c_float, _V, _V, _V, _V, _V,
                                        _V, _V]
_lib.oda_recall_gate_static.restype = ctypes.c_int
_lib.oda_commit_workspace_size.argtypes = [_P(AttnShape), _P(ctypes.c_size_t)]
_lib.oda_commit_workspace_size.restype = ctypes.c_int
_lib.oda_commit_kv.argtypes = [_P(AttnShape), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
_lib.oda_commit_kv.restype = ctypes.c_int
_lib.oda_ring_elements.argtypes = [_P(AttnShape), ctypes.c_int32, ctypes.c_int32, _P(ctypes.c_int64)]
_lib.oda_ring_elements.restype = ctypes.c_int
_lib.oda_ring_fill.argtypes = [_P(AttnShape), _V, _V, _V, _V, ctypes.c_int32, ctypes.c_int32, _V, _V, _V]
_lib.oda_ring_fill.restype = ctypes.c_int
_lib.oda_local_decode_attn_ring.argtypes = [_P(AttnShape), _P(AttnInputs), _V, _V, ctypes.c_int32, ctypes.c_int32,
                                            _V, _V, _V, ctypes.c_size_t, _V]
_lib.oda_local_decode_attn_ring.restype = ctypes.c_int
_lib.oda_commit_kv_ring.argtypes = [_P(AttnShape), _V, _V, _V, _V, _V, _V, _V, _V, _V, ctypes.c_int32, _V,
                                    ctypes.c_size_t, _V, _V, ctypes.c_int32, ctypes.c_int32, _V]
_lib.oda_commit_kv_ring.restype = ctypes.c_int
_lib.oda_dense_bf16.argtypes = [_P(DenseDesc), ctypes.c_int32, _V, _V, _V, _V, _V, _V]
_lib.oda_dense_bf16.restype = ctypes.c_int
_lib.oda_qk_norm_rope.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _V, _V, _V,
                                  ctypes.c_float, ctypes.c_double, _V, _V, _V, _V, _V, _V, _V]
_lib.oda_qk_norm_rope.restype = ctypes.c_int
_lib.oda_embed_bf16.argtypes = [_V, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _V, _V, _V]
_lib.oda_embed_bf16.restype = ctypes.c_int
_lib.oda_copy_rows.argtypes = [ctypes.c_int32, ctypes.c_int32, _V, _V, _V, _V, _V]
_lib.oda_copy_rows.restype = ctypes.c_int
_lib.oda_rms_norm_rows.argtypes = [ctypes.c_int32, ctypes.c_int32, _V, _V, ctypes.c_float, _V, _V, _V, _V]
_lib.oda_rms_norm_rows.restype = ctypes.c_int
_lib.oda_argmax.argtypes = [ctypes.c_int32, ctypes.c_int32, _V, _V, _V]
_lib.oda_argmax.restype = ctypes.c_int
_lib.oda_stream_read.argtypes = [_V, ctypes.c_size_t, _V, ctypes.c_int32, _V]
_lib.oda_stream_read.restype = ctypes.c_int
_lib.oda_status_string.argtypes = [ctypes.c_int]
_lib.oda_status_string.restype = ctypes.c_char_p
_lib.oda_last_error.argtypes = []
_lib.oda_last_error.restype = ctypes.c_char_p


def status_string(status: int) -> str:
    return _lib.oda_status_string(status).decode()


def last_error() -> str:
    return _lib.oda_last_error().decode()


def _check(status: int) -> None:
    if status != ODA_OK:
        raise OdaError(status, last_error())


def _ptr(t) -> int | None:
    """Device (or host) address of a tensor, None for None; a plain int passes through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# descriptors
# ---------------------------------------------------------------------------

@dataclass
class Shape:
    num_layers: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    max_blocks_per_seq: int
    max_seq_len: int
    num_blocks: int
    split_blocks: int = 0
    block_size: int = 16
    layer_stride_kv: int = 0

    def c(self) -> AttnShape:
        return AttnShape(self.num_layers, self.batch, self.num_q_heads, self.num_kv_heads, self.head_dim,
                         self.block_size, self.max_blocks_per_seq, self.max_seq_len, self.num_blocks,
                         self.split_blocks, 0, self.layer_stride_kv)


def inputs(q, k_cache, v_cache, block_table, seq_lens, scale, k_cur=None, v_cur=None) -> AttnInputs:
    """The C struct of device pointers; it keeps the tensors alive as long as it lives."""
    s = AttnInputs(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens),
                   _ptr(k_cur), _ptr(v_cur), float(scale))
    s._keep = (q, k_cache, v_cache, block_table, seq_lens, k_cur, v_cur)
    return s


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI, without the oda_ prefix)
# ---------------------------------------------------------------------------

def attn_workspace_size(shape: Shape, n_sink: int, window: int) -> int:
    out = ctypes.c_size_t(0)
    _check(_lib.oda_attn_workspace_size(ctypes.byref(shape.c()), n_sink, window, ctypes.byref(out)))
    return out.value


def local_decode_attn(shape: Shape, inp: AttnInputs, n_sink: int, window: int, out, lse, workspace,
                      workspace_bytes: int | None = None, stream=None) -> None:
    wb = workspace.numel() * workspace.element_size() if workspace_bytes is None and workspace is not None \
        else (workspace_bytes or 0)
    _check(_lib.oda_local_decode_attn(ctypes.byref(shape.c()), ctypes.byref(inp), n_sink, window, _ptr(out),
                                      _ptr(lse), _ptr(workspace), wb, _stream(stream)))


def full_decode_attn(shape: Shape, inp: AttnInputs, native_window: int, flags, work_list, n_work, out, lse,
                     workspace, workspace_bytes: int | None = None, stream=None) -> None:
    wb = workspace.numel() * workspace.element_size() if workspace_bytes is None and workspace is not None \
        else (workspace_bytes or 0)
    _check(_lib.oda_full_decode_attn(ctypes.byref(shape.c()), ctypes.byref(inp), native_window, _ptr(flags),
                                     _ptr(work_list), _ptr(n_work), _ptr(out), _ptr(lse), _ptr(workspace), wb,
                                     _stream(stream)))


def gate_param_count(kind: int, d_model: int, d_hidden: int) -> int:
    out = ctypes.c_int64(0)
    _check(_lib.oda_gate_param_count(kind, d_model, d_hidden, ctypes.byref(out)))
    return out.value


def gate_desc(kind: int, d_model: int, d_hidden: int, params, rms_eps: float = 1e-6) -> GateDesc:
    """The C gate description; it keeps the parameter tensor alive as long as it lives."""
    s = GateDesc(kind, d_model, d_hidden, float(rms_eps), _ptr(params))
    s._keep = params
    return s


def gate_workspace_size(gate: GateDesc, batch: int) -> int:
    out = ctypes.c_size_t(0)
    _check(_lib.oda_gate_workspace_size(ctypes.byref(gate), batch, ctypes.byref(out)))
    return out.value


def recall_gate(gate: GateDesc, batch: int, h_prev, emb, h_local, tau: float, forced, score, flags, work_list,
                n_work, recall_counter, workspace, workspace_bytes: int | None = None, stream=None) -> None:
    wb = workspace.numel() * workspace.element_size() if workspace_bytes is None and workspace is not None \
        else (workspace_bytes or 0)
    _check(_lib.oda_recall_gate(ctypes.byref(gate), batch, _ptr(h_prev), _ptr(emb), _ptr(h_local),
                                float(tau), _ptr(forced), _ptr(score), _ptr(flags), _ptr(work_list),
                                _ptr(n_work), _ptr(recall_counter), _ptr(workspace), wb, _stream(stream)))


def recall_gate_static(gate: GateDesc, batch: int, h_prev, emb, h_local, tau: float, forced, score, flags, work_list,
                       n_work, recall_counter, stream=None) -> None:
    """oda_recall_gate with the library's own static workspace (no allocation)."""
    _check(_lib.oda_recall_gate_static(ctypes.byref(gate), batch, _ptr(h_prev), _ptr(emb), _ptr(h_local),
                                       float(tau), _ptr(forced), _ptr(score), _ptr(flags), _ptr(work_list),
                                       _ptr(n_work), _ptr(recall_counter), _stream(stream)))


def commit_workspace_size(shape: Shape) -> int:
    out = ctypes.c_size_t(0)
    _check(_lib.oda_commit_workspace_size(ctypes.byref(shape.c()), ctypes.byref(out)))
    return out.value


def commit_kv(shape: Shape, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full=None, v_full=None,
              flags=None, advance: bool = True, workspace=None, workspace_bytes: int | None = None,
              stream=None) -> None:
    _check(_lib.oda_commit_kv(ctypes.byref(shape.c()), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                              _ptr(seq_lens), _ptr(k_local), _ptr(v_local), _ptr(k_full), _ptr(v_full),
                              _ptr(flags), 1 if advance else 0, _ptr(workspace),
                              _nbytes(workspace, workspace_bytes), _stream(stream)))


def ring_elements(shape: Shape, n_sink: int, window: int) -> int:
    out = ctypes.c_int64(0)
    _check(_lib.oda_ring_elements(ctypes.byref(shape.c()), n_sink, window, ctypes.byref(out)))
    return out.value


def ring_fill(shape: Shape, k_cache, v_cache, block_table, seq_lens, n_sink: int, window: int, k_ring, v_ring,
              stream=None) -> None:
    _check(_lib.oda_ring_fill(ctypes.byref(shape.c()), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                              _ptr(seq_lens), n_sink, window, _ptr(k_ring), _ptr(v_ring), _stream(stream)))


def local_decode_attn_ring(shape: Shape, inp: AttnInputs, k_ring, v_ring, n_sink: int, window: int, out, lse,
                           workspace, workspace_bytes: int | None = None, stream=None) -> None:
    _check(_lib.oda_local_decode_attn_ring(ctypes.byref(shape.c()), ctypes.byref(inp), _ptr(k_ring), _ptr(v_ring),
                                           n_sink, window, _ptr(out), _ptr(lse), _ptr(workspace),
                                           _nbytes(workspace, workspace_bytes), _stream(stream)))


def commit_kv_ring(shape: Shape, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full=None,
                   v_full=None, flags=None, advance: bool = True, workspace=None, k_ring=None, v_ring=None,
                   n_sink: int = 0, window: int = 1, workspace_bytes: int | None = None, stream=None) -> None:
    _check(_lib.oda_commit_kv_ring(ctypes.byref(shape.c()), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                   _ptr(seq_lens), _ptr(k_local), _ptr(v_local), _ptr(k_full), _ptr(v_full),
                                   _ptr(flags), 1 if advance else 0, _ptr(workspace),
                                   _nbytes(workspace, workspace_bytes), _ptr(k_ring), _ptr(v_ring), n_sink, window,
                                   _stream(stream)))


def dense_desc(in_features: int, out_features: int, mode: int, weight, norm_gain=None,
               rms_eps: float = 1e-6) -> DenseDesc:
    """The C dense-layer description; it keeps the weight and gain tensors alive."""
    s = DenseDesc(in_features, out_features, mode, float(rms_eps), _ptr(weight), _ptr(norm_gain))
    s._keep = (weight, norm_gain)
    return s


def dense_bf16(desc: DenseDesc, batch: int, x, residual, y, work_list=None, n_work=None, stream=None) -> None:
    _check(_lib.oda_dense_bf16(ctypes.byref(desc), batch, _ptr(x), _ptr(residual), _ptr(y), _ptr(work_list),
                               _ptr(n_work), _stream(stream)))


def qk_norm_rope(batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int, qkv, q_gain, k_gain,
                 rms_eps: float, rope_theta: float, seq_lens, q_out, k_out, v_out, work_list=None, n_work=None,
                 stream=None) -> None:
    _check(_lib.oda_qk_norm_rope(batch, num_q_heads, num_kv_heads, head_dim, _ptr(qkv), _ptr(q_gain),
                                 _ptr(k_gain), float(rms_eps), float(rope_theta), _ptr(seq_lens), _ptr(q_out),
                                 _ptr(k_out), _ptr(v_out), _ptr(work_list), _ptr(n_work), _stream(stream)))


def embed_bf16(table, vocab: int, d_model: int, batch: int, tokens, x, stream=None) -> None:
    _check(_lib.oda_embed_bf16(_ptr(table), vocab, d_model, batch, _ptr(tokens), _ptr(x), _stream(stream)))


def copy_rows(batch: int, row_len: int, src, dst, work_list=None, n_work=None, stream=None) -> None:
    _check(_lib.oda_copy_rows(batch, row_len, _ptr(src), _ptr(dst), _ptr(work_list), _ptr(n_work),
                              _stream(stream)))


def rms_norm_rows(batch: int, row_len: int, x, gain, rms_eps: float, y, work_list=None, n_work=None,
                  stream=None) -> None:
    _check(_lib.oda_rms_norm_rows(batch, row_len, _ptr(x), _ptr(gain), float(rms_eps), _ptr(y), _ptr(work_list),
                                  _ptr(n_work), _stream(stream)))


def argmax(batch: int, n: int, x, index, stream=None) -> None:
    _check(_lib.oda_argmax(batch, n, _ptr(x), _ptr(index), _stream(stream)))


def stream_read(src, nbytes: int, sink, groups: int = 0, stream=None) -> None:
    """Measurement aid: read nbytes of src once (the streaming-read ceiling)."""
    _check(_lib.oda_stream_read(_ptr(src), int(nbytes), _ptr(sink), groups, _stream(stream)))


# ---------------------------------------------------------------------------
# pre-marshalled calls (for tight launch loops: no per-call conversion)
# ---------------------------------------------------------------------------

class Call:
    """One entry-point call with every argument already converted."""
    __slots__ = ("fn", "args", "keep")

    def __init__(self, fn, args, keep):
        self.fn, self.args, self.keep = fn, args, keep

    def __call__(self) -> None:
        st = self.fn(*self.args)
        if st != ODA_OK:
            raise OdaError(st, last_error())


def _nbytes(ws, given):
    if given is not None:
        return given
    return 0 if ws is None else ws.numel() * ws.element_size()


def prepare_local(shape: Shape, inp: AttnInputs, n_sink: int, window: int, out, lse, workspace,
                  workspace_bytes: int | None = None, stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), ctypes.byref(inp), n_sink, window, _ptr(out), _ptr(lse), _ptr(workspace),
            _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_local_decode_attn, args, (cs, inp, out, lse, workspace))


def prepare_local_ring(shape: Shape, inp: AttnInputs, k_ring, v_ring, n_sink: int, window: int, out, lse, workspace,
                       workspace_bytes: int | None = None, stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), ctypes.byref(inp), _ptr(k_ring), _ptr(v_ring), n_sink, window, _ptr(out), _ptr(lse),
            _ptr(workspace), _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_local_decode_attn_ring, args, (cs, inp, k_ring, v_ring, out, lse, workspace))


def qkv_prep(qkv, q_gain, k_gain, rms_eps: float, rope_theta: float, k_out=None, v_out=None) -> QkvPrep:
    """The C struct of a fused call's current-token preparation; it keeps the tensors alive."""
    s = QkvPrep(_ptr(qkv), _ptr(q_gain), _ptr(k_gain), float(rms_eps), float(rope_theta), _ptr(k_out), _ptr(v_out))
    s._keep = (qkv, q_gain, k_gain, k_out, v_out)
    return s


def prepare_local_qkv(shape: Shape, inp: AttnInputs, prep: QkvPrep, n_sink: int, window: int, out, lse, workspace,
                      workspace_bytes: int | None = None, stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), ctypes.byref(inp), ctypes.byref(prep), n_sink, window, _ptr(out), _ptr(lse),
            _ptr(workspace), _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_local_decode_attn_qkv, args, (cs, inp, prep, out, lse, workspace))


def prepare_full_qkv(shape: Shape, inp: AttnInputs, prep: QkvPrep, native_window: int, flags, work_list, n_work,
                     out, lse, workspace, workspace_bytes: int | None = None, stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), ctypes.byref(inp), ctypes.byref(prep), native_window, _ptr(flags), _ptr(work_list),
            _ptr(n_work), _ptr(out), _ptr(lse), _ptr(workspace), _nbytes(workspace, workspace_bytes),
            _stream(stream))
    return Call(_lib.oda_full_decode_attn_qkv, args, (cs, inp, prep, flags, work_list, n_work, out, lse, workspace))


def prepare_full(shape: Shape, inp: AttnInputs, native_window: int, flags, work_list, n_work, out, lse,
                 workspace, workspace_bytes: int | None = None, stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), ctypes.byref(inp), native_window, _ptr(flags), _ptr(work_list), _ptr(n_work),
            _ptr(out), _ptr(lse), _ptr(workspace), _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_full_decode_attn, args, (cs, inp, flags, work_list, n_work, out, lse, workspace))


def prepare_gate(gate: GateDesc, batch: int, h_prev, emb, h_local, tau: float, forced, score, flags, work_list,
                 n_work, recall_counter, workspace, workspace_bytes: int | None = None, stream=None) -> Call:
    args = (ctypes.byref(gate), batch, _ptr(h_prev), _ptr(emb), _ptr(h_local), float(tau), _ptr(forced),
            _ptr(score), _ptr(flags), _ptr(work_list), _ptr(n_work), _ptr(recall_counter), _ptr(workspace),
            _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_recall_gate, args, (gate, h_prev, emb, h_local, forced, score, flags, work_list, n_work,
                                            recall_counter, workspace))


def prepare_commit(shape: Shape, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full=None,
                   v_full=None, flags=None, advance: bool = True, workspace=None, workspace_bytes: int | None = None,
                   stream=None) -> Call:
    cs = shape.c()
    args = (ctypes.byref(cs), _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(seq_lens), _ptr(k_local),
            _ptr(v_local), _ptr(k_full), _ptr(v_full), _ptr(flags), 1 if advance else 0, _ptr(workspace),
            _nbytes(workspace, workspace_bytes), _stream(stream))
    return Call(_lib.oda_commit_kv, args, (cs, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full,
                                          v_full, flags, workspace))


def prepare_dense(desc: DenseDesc, batch: int, x, residual, y, work_list=None, n_work=None, stream=None) -> Call:
    args = (ctypes.byref(desc), batch, _ptr(x), _ptr(residual), _ptr(y), _ptr(work_list), _ptr(n_work),
            _stream(stream))
    return Call(_lib.oda_dense_bf16, args, (desc, x, residual, y, work_list, n_work))


def prepare_qk_norm_rope(batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int, qkv, q_gain, k_gain,
                         rms_eps: float, rope_theta: float, seq_lens, q_out, k_out, v_out, work_list=None,
                         n_work=None, stream=None) -> Call:
    args = (batch, num_q_heads, num_kv_heads, head_dim, _ptr(qkv), _ptr(q_gain), _ptr(k_gain), float(rms_eps),
            float(rope_theta), _ptr(seq_lens), _ptr(q_out), _ptr(k_out), _ptr(v_out), _ptr(work_list),
            _ptr(n_work), _stream(stream))
    return Call(_lib.oda_qk_norm_rope, args, (qkv, q_gain, k_gain, seq_lens, q_out, k_out, v_out, work_list,
                                              n_work))


def prepare_embed(table, vocab: int, d_model: int, batch: int, tokens, x, stream=None) -> Call:
    args = (_ptr(table), vocab, d_model, batch, _ptr(tokens), _ptr(x), _stream(stream))
    return Call(_lib.oda_embed_bf16, args, (table, tokens, x))


def prepare_copy_rows(batch: int, row_len: int, src, dst, work_list=None, n_work=None, stream=None) -> Call:
    args = (batch, row_len, _ptr(src), _ptr(dst), _ptr(work_list), _ptr(n_work), _stream(stream))
    return Call(_lib.oda_copy_rows, args, (src, dst, work_list, n_work))


def prepare_rms_norm_rows(batch: int, row_len: int, x, gain, rms_eps: float, y, work_list=None, n_work=None,
                          stream=None) -> Call:
    args = (batch, row_len, _ptr(x), _ptr(gain), float(rms_eps), _ptr(y), _ptr(work_list), _ptr(n_work),
            _stream(stream))
    return Call(_lib.oda_rms_norm_rows, args, (x, gain, y, work_list, n_work))


def prepare_argmax(batch: int, n: int, x, index, stream=None) -> Call:
    args = (batch, n, _ptr(x), _ptr(index), _stream(stream))
    return Call(_lib.oda_argmax, args, (x, index))


def prepare_stream_read(src, nbytes: int, sink, groups: int = 0, stream=None) -> Call:
    args = (_ptr(src), int(nbytes), _ptr(sink), groups, _stream(stream))
    return Call(_lib.oda_stream_read, args, (src, sink))
