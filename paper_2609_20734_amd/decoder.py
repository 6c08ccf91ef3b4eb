"""A whole ODA decode step on a synthetic decoder, composed from the C-ABI
entry points (every operation runs in liboda's HIP kernels; this module only
prepares the calls).

Per step (Alg. 1 with the commit of App. A.5):

  local stage   embed the step's tokens; the Local forward (every layer:
                QKV, q/k norm + rotary, Local attention with the Local
                candidate, output projection, SwiGLU MLP); the final RMSNorm
                of the Local hidden state (h^L_t, §2.1); the recall gate on
                (h_{t-1}, E(x_t), h^L_t), writing flags and the compacted list
  retry stage   the Full forward from the same pre-step history for the listed
                requests only, then their final hidden rows replace the Local
                ones (App. A.5: only the selected state is kept)
  output stage  the final RMSNorm of the selected state (this is h_{t-1} of
                the next step's gate, App. A.5) and the vocabulary projection
                of it, greedy token, the fused commit of the selected
                candidates of every layer

Native Full (always Full, no gate) and standalone Local (no gate, no retry)
use the same pieces.  Stages are lists of pre-marshalled calls, so they can be
launched eagerly or captured as HIP graphs.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

from . import _lib as P


@dataclass(frozen=True)
class DecoderShape:
    num_layers: int
    d_model: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 1e6

    @property
    def qkv_dim(self) -> int:
        return (self.num_q_heads + 2 * self.num_kv_heads) * self.head_dim

    def weight_bytes(self) -> int:
        """bf16 weight bytes one forward streams (vocabulary projection included)."""
        d, L = self.d_model, self.num_layers
        per_layer = (self.qkv_dim * d + d * self.num_q_heads * self.head_dim + 3 * self.d_ffn * d) * 2
        return L * per_layer + self.vocab * d * 2


# Qwen3-1.7B-shaped backbone (the model of the paper's throughput table):
# 28 layers, d = 2048, 16 query / 8 KV heads of 128, SwiGLU 6144, 151,936 tokens.
QWEN3_1_7B = DecoderShape(28, 2048, 16, 8, 128, 6144, 151936)


class Decoder:
    """Device buffers and prepared calls of one decoder over a paged cache.

    weights: dict of device tensors named as oda_synth.decoder_tensor_specs
    (bf16 weights, fp32 gains); cache, table and lengths as the attention ABI
    takes them; gate: a GateDesc for the recall head (None: no gate);
    prescribed: the gate takes its flags from `self.forced` (int32 [B], written
    before each step) instead of comparing the score with tau (App. B.7);
    fused_prep: each attention call builds its query and candidate K/V from the
    QKV projection itself (oda_*_decode_attn_qkv, bit-identical), else
    oda_qk_norm_rope runs as a launch of its own before it."""

    def __init__(self, shape: DecoderShape, weights: dict, batch: int, k_cache, v_cache, block_table, seq_lens,
                 max_blocks_per_seq: int, max_seq_len: int, num_blocks: int, n_sink: int, window: int,
                 gate=None, tau: float = 0.0, prescribed: bool = False, split_blocks: int = 0,
                 fused_prep: bool = True):
        import torch
        s, B = shape, batch
        dev = k_cache.device
        self.shape, self.B, self.w = s, B, weights
        self.k_cache, self.v_cache, self.table, self.seq_lens = k_cache, v_cache, block_table, seq_lens
        self.n_sink, self.window = n_sink, window
        self.fused_prep = fused_prep
        f32 = dict(dtype=torch.float32, device=dev)
        bf = dict(dtype=torch.bfloat16, device=dev)
        i32 = dict(dtype=torch.int32, device=dev)
        L, d, Hq, Hkv, D = s.num_layers, s.d_model, s.num_q_heads, s.num_kv_heads, s.head_dim
        self.tokens = torch.zeros(B, **i32)            # the step's tokens (written before each step)
        self.emb = torch.zeros(B, d, **f32)
        self.h = torch.zeros(B, d, **f32)               # selected state (Local stream, then selected)
        self.h_full = torch.zeros(B, d, **f32)          # Full retry stream
        self.h_prev = torch.zeros(B, d, **f32)         # final-normalised selected state of the last step
        self.h_local = torch.zeros(B, d, **f32)        # final-normalised Local state (the gate's h^L_t)
        self.qkv = torch.zeros(B, s.qkv_dim, **f32)
        self.q = torch.zeros(B, Hq, D, **bf)
        self.attn = torch.zeros(B, Hq * D, **f32)
        self.lse = torch.zeros(B, Hq, **f32)
        self.mlp = torch.zeros(B, s.d_ffn, **f32)
        self.logits = torch.zeros(B, s.vocab, **f32)
        self.next_token = torch.zeros(B, **i32)
        self.k_loc = torch.zeros(L, B, Hkv, D, **bf)
        self.v_loc = torch.zeros(L, B, Hkv, D, **bf)
        self.k_full = torch.zeros(L, B, Hkv, D, **bf)
        self.v_full = torch.zeros(L, B, Hkv, D, **bf)
        self.score = torch.zeros(B, **f32)
        self.flags = torch.zeros(B, **i32)
        self.work = torch.zeros(B, **i32)
        self.n_work = torch.zeros(1, **i32)
        self.counter = torch.zeros(1, dtype=torch.int64, device=dev)
        self.gate, self.tau = gate, tau
        self.forced = torch.zeros(B, **i32) if prescribed else None
        self.ws_gate = None if gate is None else torch.zeros(P.gate_workspace_size(gate, B), dtype=torch.uint8,
                                                             device=dev)
        # one-layer attention calls: the layer's slices of the caches and candidates
        self.attn_shape = P.Shape(1, B, Hq, Hkv, D, max_blocks_per_seq, max_seq_len, num_blocks, split_blocks)
        self.ws_local = torch.zeros(max(256, P.attn_workspace_size(self.attn_shape, n_sink, window)),
                                    dtype=torch.uint8, device=dev)
        self.ws_full = torch.zeros(max(256, P.attn_workspace_size(self.attn_shape, 0, 0)), dtype=torch.uint8,
                                   device=dev)
        self.ws_commit = torch.zeros(P.commit_workspace_size(self.commit_shape()), dtype=torch.uint8, device=dev)
        self.scale = 1.0 / math.sqrt(D)
        w = weights
        self.d_qkv = [P.dense_desc(d, s.qkv_dim, P.DENSE_PLAIN, w["w_qkv"][l], w["attn_norm"][l], s.rms_eps)
                      for l in range(L)]
        self.d_o = [P.dense_desc(Hq * D, d, P.DENSE_PLAIN, w["w_o"][l]) for l in range(L)]
        self.d_gu = [P.dense_desc(d, s.d_ffn, P.DENSE_SWIGLU, w["w_gu"][l], w["mlp_norm"][l], s.rms_eps)
                     for l in range(L)]
        self.d_down = [P.dense_desc(s.d_ffn, d, P.DENSE_PLAIN, w["w_down"][l]) for l in range(L)]
        # the vocabulary projection reads the final-normalised state (h_prev after the output stage's norm)
        self.d_vocab = P.dense_desc(d, s.vocab, P.DENSE_PLAIN, w["embed"])

    # -- stages ---------------------------------------------------------------
    def _forward(self, h, k_cand, v_cand, branch: str, listed: bool):
        """Calls of one forward on stream h (branch "local" or "full")."""
        s, B = self.shape, self.B
        wl = (self.work, self.n_work) if listed else (None, None)
        calls = []
        for l in range(s.num_layers):
            calls.append(P.prepare_dense(self.d_qkv[l], B, h, None, self.qkv, *wl))
            if self.fused_prep:
                prep = P.qkv_prep(self.qkv, self.w["q_norm"][l], self.w["k_norm"][l], s.rms_eps, s.rope_theta,
                                  k_cand[l], v_cand[l])
                inp = P.inputs(None, self.k_cache[l], self.v_cache[l], self.table, self.seq_lens, self.scale)
                if branch == "local":
                    calls.append(P.prepare_local_qkv(self.attn_shape, inp, prep, self.n_sink, self.window, self.attn,
                                                     self.lse, self.ws_local))
                else:
                    calls.append(P.prepare_full_qkv(self.attn_shape, inp, prep, 0, None, *wl, self.attn, self.lse,
                                                    self.ws_full))
            else:
                calls.append(P.prepare_qk_norm_rope(B, s.num_q_heads, s.num_kv_heads, s.head_dim, self.qkv,
                                                    self.w["q_norm"][l], self.w["k_norm"][l], s.rms_eps,
                                                    s.rope_theta, self.seq_lens, self.q, k_cand[l], v_cand[l], *wl))
                inp = P.inputs(self.q, self.k_cache[l], self.v_cache[l], self.table, self.seq_lens, self.scale,
                               k_cand[l], v_cand[l])
                if branch == "local":
                    calls.append(P.prepare_local(self.attn_shape, inp, self.n_sink, self.window, self.attn,
                                                 self.lse, self.ws_local))
                else:
                    calls.append(P.prepare_full(self.attn_shape, inp, 0, None, *wl, self.attn, self.lse,
                                                self.ws_full))
            calls.append(P.prepare_dense(self.d_o[l], B, self.attn, h, h, *wl))
            calls.append(P.prepare_dense(self.d_gu[l], B, h, None, self.mlp, *wl))
            calls.append(P.prepare_dense(self.d_down[l], B, self.mlp, h, h, *wl))
        return calls

    def _input(self):
        s, B = self.shape, self.B
        return [P.prepare_embed(self.w["embed"], s.vocab, s.d_model, B, self.tokens, self.emb),
                P.prepare_copy_rows(B, s.d_model, self.emb, self.h)]

    def _output(self, k_full=None, v_full=None, flags=None):
        s, B = self.shape, self.B
        return [P.prepare_rms_norm_rows(B, s.d_model, self.h, self.w["final_norm"], s.rms_eps, self.h_prev),
                P.prepare_dense(self.d_vocab, B, self.h_prev, None, self.logits),
                P.prepare_argmax(B, s.vocab, self.logits, self.next_token),
                P.prepare_commit(self.commit_shape(), self.k_cache, self.v_cache, self.table, self.seq_lens,
                                 self.k_loc, self.v_loc, k_full, v_full, flags, True, self.ws_commit)]

    def commit_shape(self) -> P.Shape:
        a = self.attn_shape
        return P.Shape(self.shape.num_layers, a.batch, a.num_q_heads, a.num_kv_heads, a.head_dim,
                       a.max_blocks_per_seq, a.max_seq_len, a.num_blocks, a.split_blocks)

    def oda_stages(self):
        """(local stage, retry stage, output stage) of one ODA step."""
        s, B = self.shape, self.B
        assert self.gate is not None
        local = self._input() + self._forward(self.h, self.k_loc, self.v_loc, "local", False)
        local.append(P.prepare_rms_norm_rows(B, s.d_model, self.h, self.w["final_norm"], s.rms_eps, self.h_local))
        local.append(P.prepare_gate(self.gate, B, self.h_prev, self.emb, self.h_local, self.tau, self.forced,
                                    self.score, self.flags, self.work, self.n_work, self.counter, self.ws_gate))
        retry = [P.prepare_copy_rows(B, s.d_model, self.emb, self.h_full, self.work, self.n_work)]
        retry += self._forward(self.h_full, self.k_full, self.v_full, "full", True)
        retry.append(P.prepare_copy_rows(B, s.d_model, self.h_full, self.h, self.work, self.n_work))
        out = self._output(self.k_full, self.v_full, self.flags)
        return local, retry, out

    def full_stages(self):
        """Native Full: every layer over its whole history, no gate."""
        return self._input() + self._forward(self.h, self.k_loc, self.v_loc, "full", False), [], self._output()

    def local_stages(self):
        """Standalone Local: every layer over S^L, no gate, no retry."""
        return self._input() + self._forward(self.h, self.k_loc, self.v_loc, "local", False), [], self._output()


def run(calls) -> None:
    for c in calls:
        c()
