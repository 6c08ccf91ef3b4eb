"""Algorithmic bytes of one decode step.  TEST INFRASTRUCTURE.

The byte analogue of the cost model of App. A.6 (Eq. speed-general with the
history-independent terms B = O = 0) and of the operation ledger of App. B.7:
KV bytes scale with KV heads, so each attended position costs Hkv * 4D bytes
(bf16 K and V) per layer.  Only the method's own reads and writes count: q,
the attended K/V rows, the block-table entries of the visited blocks, the
gate's fp32 weights and inputs, and the fp32 outputs.  Scratch traffic of an
implementation (split partials) is excluded.
"""
from __future__ import annotations

import numpy as np

from . import attention as A
from . import gate as Gt

BLOCK_SIZE = 16


def attention_bytes(seq_lens, positions_of, num_layers, num_q_heads, num_kv_heads, head_dim,
                    requests=None, with_lse=True):
    """Bytes of one attention pass over ``requests`` (default: all):
    returns dict kv, q, out, table, total."""
    seq_lens = np.asarray(seq_lens)
    reqs = range(len(seq_lens)) if requests is None else requests
    kv = q = out = table = 0
    for b in reqs:
        n = int(seq_lens[b])
        S = positions_of(n)
        kv += len(S) * num_kv_heads * 4 * head_dim * num_layers
        q += num_q_heads * head_dim * 2 * num_layers
        out += num_q_heads * (head_dim + (1 if with_lse else 0)) * 4 * num_layers
        table += len(np.unique(S // BLOCK_SIZE)) * 4
    return dict(kv=kv, q=q, out=out, table=table, total=kv + q + out + table)


def gate_bytes(kind: str, batch: int, d_model: int, d_hidden: int):
    """fp32 head weights + the inputs it reads (3 rows per request for the
    App. A.2 head, h^L only for the MLP) + score/flag/list writes."""
    shapes = Gt.paper_head_shapes(d_model, d_hidden) if kind == "paper" else Gt.mlp_shapes(d_model, d_hidden)
    w = Gt.param_count(shapes) * 4
    inputs = batch * (3 if kind == "paper" else 1) * d_model * 4
    outs = batch * 4 * 3 + 4 + 8
    return dict(weights=w, inputs=inputs, outputs=outs, total=w + inputs + outs)


def step_bytes(seq_lens, flags, n_sink, window, native_window, num_layers, num_q_heads,
               num_kv_heads, head_dim, gate_kind, d_model, d_hidden):
    """Bytes(rho) of one step: Local for all requests, the gate, Full for the
    flagged ones.  Returns dict local, gate, full, total."""
    loc = attention_bytes(seq_lens, lambda n: A.local_set(n, n_sink, window), num_layers,
                          num_q_heads, num_kv_heads, head_dim)
    gt = gate_bytes(gate_kind, len(seq_lens), d_model, d_hidden)
    flagged = list(np.flatnonzero(np.asarray(flags)))
    full = attention_bytes(seq_lens, lambda n: A.native_window_set(n, native_window), num_layers,
                           num_q_heads, num_kv_heads, head_dim, requests=flagged)
    return dict(local=loc["total"], gate=gt["total"], full=full["total"],
                total=loc["total"] + gt["total"] + full["total"])


def always_full_bytes(seq_lens, native_window, num_layers, num_q_heads, num_kv_heads, head_dim):
    """Bytes_Full: the native Full pass for every request, no Local, no gate."""
    return attention_bytes(seq_lens, lambda n: A.native_window_set(n, native_window), num_layers,
                           num_q_heads, num_kv_heads, head_dim)["total"]
