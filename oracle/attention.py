"""Decode attention, fp64, by definition.  TEST INFRASTRUCTURE (see package doc).

Positions are 0-based here: the paper's position t (1-based, §2.1) is our
n = t attended positions 0..n-1, the last of which (n-1) is the current
token.
"""
from __future__ import annotations

import numpy as np

BLOCK_SIZE = 16


def bf16_to_f64(bits) -> np.ndarray:
    """Widen raw bf16 bits (uint16) to float64.  Exact."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16)).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# access sets  (§2.1, access-set equation)
# ---------------------------------------------------------------------------

def full_set(n: int) -> np.ndarray:
    """S^F: every position 1..t (0-based: 0..n-1)."""
    return np.arange(n, dtype=np.int64)


def local_set(n: int, n_sink: int, window: int) -> np.ndarray:
    """S^L: the first min(s, t) positions united with the recent window
    max(1, t-w+1)..t, which includes the current token (§2.1).  As a set, so a
    position in both parts counts once.  0-based."""
    sinks = set(range(0, min(n_sink, n)))
    recent = set(range(max(0, n - window), n))
    return np.array(sorted(sinks | recent), dtype=np.int64)


def native_window_set(n: int, window: int) -> np.ndarray:
    """A natively sliding-window layer's own set: the last ``window``
    positions, no sinks (native layers keep their computation, §2.1)."""
    if window <= 0:
        return full_set(n)
    return local_set(n, 0, window)


# ---------------------------------------------------------------------------
# paged cache access (ABI layouts)
# ---------------------------------------------------------------------------

def key_rows(k_cache, block_table, layer, b, kv_head, positions) -> np.ndarray:
    """K rows for the given positions.  k_cache: uint16 [L][NB][Hkv][D/8][16][8];
    logical block i of request b lives in physical block block_table[b][i],
    position p sits in slot p % 16 of logical block p // 16."""
    pos = np.asarray(positions, dtype=np.int64)
    phys = block_table[b, pos // BLOCK_SIZE].astype(np.int64)
    rows = k_cache[layer, phys, kv_head, :, pos % BLOCK_SIZE, :]   # [P][D/8][8]
    return bf16_to_f64(rows).reshape(len(pos), k_cache.shape[3] * k_cache.shape[5])


def value_rows(v_cache, block_table, layer, b, kv_head, positions) -> np.ndarray:
    """V rows for the given positions.  v_cache: uint16 [L][NB][Hkv][D][16]."""
    pos = np.asarray(positions, dtype=np.int64)
    phys = block_table[b, pos // BLOCK_SIZE].astype(np.int64)
    rows = v_cache[layer, phys, kv_head, :, pos % BLOCK_SIZE]      # [P][D]
    return bf16_to_f64(rows).reshape(len(pos), v_cache.shape[3])


# ---------------------------------------------------------------------------
# attention for one query head
# ---------------------------------------------------------------------------

def attend(q, K, V, scale: float):
    """Softmax attention of one query over the rows of K, V.

    z_j = scale * q.K_j;  M = max z;  p_j = exp(z_j - M);  Z = sum p;
    o = sum_j (p_j / Z) V_j;  lse = M + ln Z.   Returns (o, lse, weights).
    """
    z = scale * (K @ q)
    M = np.max(z)
    p = np.exp(z - M)
    Z = np.sum(p)
    w = p / Z
    return w @ V, M + np.log(Z), w


def decode_attention(q, k_cache, v_cache, block_table, seq_lens, positions_of, scale,
                     k_cur=None, v_cur=None, layers=None, requests=None, return_weights=False):
    """Decode attention for every (layer, request, query head).

    q: uint16 bf16 [L][B][Hq][D]; caches in the ABI layouts; positions_of(n)
    gives the attended positions of a request with n positions.  If k_cur /
    v_cur (uint16 [L][B][Hkv][D]) are given, position n-1 is the uncommitted
    current candidate taken from them instead of the cache (App. A.5).
    Query head h reads KV head h // G (contiguous GQA groups).

    Returns out f64 [L][B][Hq][D], lse f64 [L][B][Hq] (rows not requested are
    NaN) and counts int [B] (|S| per request).  With return_weights, also a
    dict (l, b, h) -> (positions, weights).
    """
    L, B, Hq, D = q.shape
    Hkv = k_cache.shape[2]
    G = Hq // Hkv
    layers = range(L) if layers is None else layers
    requests = range(B) if requests is None else requests
    out = np.full((L, B, Hq, D), np.nan)
    lse = np.full((L, B, Hq), np.nan)
    counts = np.zeros(B, dtype=np.int64)
    weights = {}
    for b in requests:
        n = int(seq_lens[b])
        S = positions_of(n)
        counts[b] = len(S)
        cached = S[S < n - 1] if k_cur is not None else S
        for l in layers:
            for g in range(Hkv):
                K = key_rows(k_cache, block_table, l, b, g, cached)
                V = value_rows(v_cache, block_table, l, b, g, cached)
                if k_cur is not None and (n - 1) in S:
                    K = np.vstack([K, bf16_to_f64(k_cur[l, b, g])[None, :]])
                    V = np.vstack([V, bf16_to_f64(v_cur[l, b, g])[None, :]])
                for h in range(g * G, (g + 1) * G):
                    o, s, w = attend(bf16_to_f64(q[l, b, h]), K, V, scale)
                    out[l, b, h] = o
                    lse[l, b, h] = s
                    if return_weights:
                        weights[(l, b, h)] = (S, w)
    if return_weights:
        return out, lse, counts, weights
    return out, lse, counts


# ---------------------------------------------------------------------------
# combining partial results (the second Local kernel's role, App. A.5)
# ---------------------------------------------------------------------------

def partial_attend(q, K, V, scale: float):
    """Unnormalised partial over one subset: (m, l, o) with m = max z,
    l = sum exp(z - m), o = sum exp(z - m) V."""
    z = scale * (K @ q)
    m = np.max(z)
    e = np.exp(z - m)
    return m, np.sum(e), e @ V


def combine_partials(parts):
    """Stable-softmax combination of partials over disjoint subsets:
    M = max m_i,  Lambda = sum l_i e^{m_i - M},
    o = sum e^{m_i - M} o_i / Lambda,  lse = M + ln Lambda."""
    M = max(m for m, _, _ in parts)
    lam = sum(l * np.exp(m - M) for m, l, _ in parts)
    o = sum(oi * np.exp(m - M) for m, _, oi in parts) / lam
    return o, M + np.log(lam)
