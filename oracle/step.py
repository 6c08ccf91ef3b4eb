"""One ODA decode step (attention part), fp64.  TEST INFRASTRUCTURE.

Alg. 1 restricted to the hot path: Local attention on the access set S^L,
the recall score, the decision, Full attention from the same pre-step history
for flagged requests only, and the selected output (App. A.5: the selected
branch's state is the one kept).
"""
from __future__ import annotations

import numpy as np

from . import attention as A
from . import gate as Gt


def decode_step(q, k_cache, v_cache, block_table, seq_lens, scale, n_sink, window,
                gate_kind, gate_params, d_model, d_hidden, eps, h_prev, emb, h_local, tau,
                forced=None, native_window=0, k_cur=None, v_cur=None, layers=None, requests=None):
    """Returns dict with out_local, lse_local, score, flags, work_list, n_work,
    out_full (NaN rows for unflagged requests), out (selected), lse (selected)."""
    local = A.decode_attention(q, k_cache, v_cache, block_table, seq_lens,
                               lambda n: A.local_set(n, n_sink, window), scale,
                               k_cur=k_cur, v_cur=v_cur, layers=layers, requests=requests)
    if gate_kind == "paper":
        score = Gt.paper_head_score(gate_params, d_model, d_hidden, eps, h_prev, emb, h_local)
    else:
        score = Gt.mlp_score(gate_params, d_model, d_hidden, h_local)
    flags = Gt.decide(score, tau, forced)
    work, n_work = Gt.compact(flags)
    req = work if requests is None else [b for b in work if b in set(requests)]
    full = A.decode_attention(q, k_cache, v_cache, block_table, seq_lens,
                              lambda n: A.native_window_set(n, native_window), scale,
                              k_cur=k_cur, v_cur=v_cur, layers=layers, requests=req)
    out = local[0].copy()
    lse = local[1].copy()
    for b in work:
        out[:, b] = full[0][:, b]
        lse[:, b] = full[1][:, b]
    return dict(out_local=local[0], lse_local=local[1], count_local=local[2],
                score=score, flags=flags.astype(np.int32), work_list=work, n_work=n_work,
                out_full=full[0], lse_full=full[1], out=out, lse=lse)


def commit(k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full, v_full, flags):
    """C_t = C_{t-1} || dC_t^{b_t} (App. A.5, commit equation), in place on host
    copies: the selected branch's candidate K/V of every layer goes to position
    n_b - 1 of request b; then every n_b advances by one.  Pure data movement."""
    L, B, Hkv, D = k_local.shape
    for b in range(B):
        pos = int(seq_lens[b]) - 1
        phys = int(block_table[b, pos // 16])
        ks, vs = (k_full, v_full) if flags[b] else (k_local, v_local)
        for l in range(L):
            for g in range(Hkv):
                k_cache[l, phys, g, :, pos % 16, :] = ks[l, b, g].reshape(D // 8, 8)
                v_cache[l, phys, g, :, pos % 16] = vs[l, b, g]
        seq_lens[b] += 1
