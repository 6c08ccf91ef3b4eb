"""Algorithmic bytes of the decode-step hot path, in closed form.

The byte analogue of the cost model of App. A.6 (speed-general equation with
B = O = 0) and of the operation ledger of App. B.7, where KV bytes scale with
KV heads: an attended position costs Hkv * 4D bytes (bf16 K and V) per layer.
Counted: q, attended K/V rows, visited block-table entries, fp32 outputs
(out + lse), the gate's fp32 weights and inputs, and its small outputs.
Split-K scratch traffic is implementation overhead and is not counted.
"""
from __future__ import annotations

BLOCK = 16


def local_count(n: int, n_sink: int, window: int) -> int:
    """|S^L| for n positions: |[0, a) U [c, n)| with a = min(s, n), c = max(0, n - w)."""
    if window <= 0:
        return n
    a = min(n_sink, n)
    c = max(0, n - window)
    return a + (n - c) - max(0, a - c)


def visited_blocks(n: int, n_sink: int, window: int) -> int:
    """Distinct 16-position blocks holding attended positions."""
    if window <= 0:
        return (n + BLOCK - 1) // BLOCK
    a = min(n_sink, n)
    c = max(0, n - window)
    sink_blocks = set(range(0, (a + BLOCK - 1) // BLOCK))
    recent_blocks = set(range(c // BLOCK, (n + BLOCK - 1) // BLOCK))
    return len(sink_blocks | recent_blocks)


def attention_bytes(seq_lens, n_sink, window, num_layers, num_q_heads, num_kv_heads, head_dim,
                    requests=None, with_lse=True) -> dict:
    reqs = range(len(seq_lens)) if requests is None else requests
    kv = q = out = table = 0
    for b in reqs:
        n = int(seq_lens[b])
        kv += local_count(n, n_sink, window) * num_kv_heads * 4 * head_dim * num_layers
        q += num_q_heads * head_dim * 2 * num_layers
        out += num_q_heads * (head_dim + (1 if with_lse else 0)) * 4 * num_layers
        table += visited_blocks(n, n_sink, window) * 4
    return dict(kv=kv, q=q, out=out, table=table, total=kv + q + out + table)


def gate_param_count(kind: str, d: int, dh: int) -> int:
    if kind == "paper":
        return 3 * (d * dh + dh + d) + (9 * dh * dh + dh) + 2 * (dh + 3 * dh * 2 * dh) + (2 * dh + 1)
    return dh * d + 2 * dh + 1


def gate_bytes(kind: str, batch: int, d: int, dh: int) -> dict:
    w = gate_param_count(kind, d, dh) * 4
    inputs = batch * (3 if kind == "paper" else 1) * d * 4
    outs = batch * 4 * 3 + 4 + 8
    return dict(weights=w, inputs=inputs, outputs=outs, total=w + inputs + outs)
