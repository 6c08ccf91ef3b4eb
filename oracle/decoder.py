"""The decoder around the hot path, fp64.  TEST INFRASTRUCTURE.

§2.1 defines the two branches as the same backbone f_theta run with different
attention access sets (S^L or S^F in every restricted layer); Alg. 1 runs the
Local forward, scores it, and reruns the whole forward with Full from the same
pre-step history when the predicate fires; App. A.5 keeps only the selected
branch's state; App. A.6 prices a step as backbone + attention + head +
output.  The paper takes the backbone from its models without restating it,
so its form here is a reading: a pre-norm decoder layer

    h  <- h + W_o . Attn(rope(rmsnorm_head(q)), rope(rmsnorm_head(k)), v)
          with q, k, v = W_qkv . RMSNorm(h)
    h  <- h + W_d . (SiLU(W_g . RMSNorm(h)) * (W_u . RMSNorm(h)))

then logits = W_vocab . RMSNorm(h) and the greedy token.  The rotary
embedding pairs dimension i with i + D/2 and turns the pair by the angle
p * theta^(-2i/D) at position p.

Precision points shared with the product path: weights are bf16 values; q,
k, v are rounded to bf16 (they are the attention's inputs, and k, v become
cache entries).  Everything else is float64.
"""
from __future__ import annotations

import numpy as np

from . import attention as A


def round_bf16(x) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned as float64.
    Values are first rounded to float32 (nearest-even), then to bf16."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = (((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out)


def bf16_bits(x) -> np.ndarray:
    """Raw bits of values that are already bf16 (as produced by round_bf16)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def rmsnorm(x, gain, eps: float):
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(gain, dtype=np.float64)


def silu(x):
    return x / (1.0 + np.exp(-x))


def dense(w_bits, x, gain=None, eps: float = 1e-6, residual=None):
    """W . x' (+ residual), x' = RMSNorm(x) with `gain`, or x itself."""
    W = A.bf16_to_f64(w_bits)
    xin = rmsnorm(x, gain, eps) if gain is not None else np.asarray(x, dtype=np.float64)
    y = xin @ W.T
    return y if residual is None else y + residual


def swiglu(w_bits, x, gain, eps: float):
    """SiLU(W_g . x') * (W_u . x'); w_bits holds the gate rows, then the up
    rows; x' = RMSNorm(x) with `gain`, or x itself (as in `dense`)."""
    W = A.bf16_to_f64(w_bits)
    F = W.shape[0] // 2
    xin = rmsnorm(x, gain, eps) if gain is not None else np.asarray(x, dtype=np.float64)
    return silu(xin @ W[:F].T) * (xin @ W[F:].T)


def rope(x, pos, theta: float):
    """Rotary embedding of the last axis (length D) at positions `pos`
    (broadcast over the leading axes): pair (i, i + D/2) turned by
    pos * theta^(-2i/D)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * theta ** (-2.0 * np.arange(half) / D)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def qk_norm_rope(qkv, Hq: int, Hkv: int, D: int, q_gain, k_gain, eps: float, theta: float, pos):
    """Split qkv [B][(Hq + 2 Hkv) D] into heads, per-head RMSNorm of q and k
    (gain None: no norm), rotary embedding at pos [B], round to bf16.
    Returns q [B][Hq][D], k [B][Hkv][D], v [B][Hkv][D] (bf16 values, float64)."""
    B = qkv.shape[0]
    heads = np.asarray(qkv, dtype=np.float64).reshape(B, Hq + 2 * Hkv, D)
    q, k, v = heads[:, :Hq], heads[:, Hq:Hq + Hkv], heads[:, Hq + Hkv:]
    if q_gain is not None:
        q = rmsnorm(q, q_gain, eps)
    if k_gain is not None:
        k = rmsnorm(k, k_gain, eps)
    p = np.asarray(pos, dtype=np.float64)[:, None]
    return round_bf16(rope(q, p, theta)), round_bf16(rope(k, p, theta)), round_bf16(v)


class Model:
    """Synthetic weights (the dict of oda_synth.decoder_weights) and shape."""

    def __init__(self, weights: dict, Hq: int, Hkv: int, D: int, eps: float = 1e-6, theta: float = 1e6):
        self.w = weights
        self.L = weights["w_qkv"].shape[0]
        self.d = weights["embed"].shape[1]
        self.V = weights["embed"].shape[0]
        self.Hq, self.Hkv, self.D = Hq, Hkv, D
        self.eps, self.theta = eps, theta

    def embed(self, tokens):
        return A.bf16_to_f64(self.w["embed"][np.asarray(tokens)])

    def forward(self, tokens, k_cache, v_cache, block_table, seq_lens, positions_of, requests=None):
        """One forward of the current token of every request in `requests`
        (default all), every layer attending over positions_of(n) of its
        cache plus the current candidate at position n - 1 (App. A.5).
        Returns (final hidden [B][d] (NaN rows for others), k_cand, v_cand
        [L][B][Hkv][D] bf16 bits)."""
        w, L, Hq, Hkv, D = self.w, self.L, self.Hq, self.Hkv, self.D
        B = len(tokens)
        req = list(range(B)) if requests is None else list(requests)
        h = np.full((B, self.d), np.nan)
        h[req] = self.embed(np.asarray(tokens)[req])
        kc = np.zeros((L, B, Hkv, D), dtype=np.uint16)
        vc = np.zeros((L, B, Hkv, D), dtype=np.uint16)
        pos = np.asarray(seq_lens, dtype=np.int64) - 1
        scale = 1.0 / np.sqrt(D)
        for l in range(L):
            qkv = dense(w["w_qkv"][l], h[req], w["attn_norm"][l], self.eps)
            q, k, v = qk_norm_rope(qkv, Hq, Hkv, D, w["q_norm"][l], w["k_norm"][l], self.eps, self.theta, pos[req])
            qb = np.zeros((1, B, Hq, D), dtype=np.uint16)
            qb[0, req] = bf16_bits(q)
            kc[l, req] = bf16_bits(k)
            vc[l, req] = bf16_bits(v)
            out = A.decode_attention(qb, k_cache[l:l + 1], v_cache[l:l + 1], block_table, seq_lens, positions_of,
                                     scale, k_cur=kc[l:l + 1], v_cur=vc[l:l + 1], requests=req)[0][0]
            attn = out[req].reshape(len(req), Hq * D)
            h[req] = dense(w["w_o"][l], attn, residual=h[req])
            m = swiglu(w["w_gu"][l], h[req], w["mlp_norm"][l], self.eps)
            h[req] = dense(w["w_down"][l], m, residual=h[req])
        return h, kc, vc

    def final_state(self, h):
        """The final normalised hidden state RMSNorm(h) with the final gain:
        the head's h^L_t for the Local branch (§2.1) and, for the selected
        branch, the state the vocabulary projection reads, which is the
        head's h_{t-1} at the next step (App. A.5)."""
        return rmsnorm(h, self.w["final_norm"], self.eps)

    def logits(self, h):
        """W_vocab . RMSNorm(h) with the vocabulary projection tied to the embedding."""
        return dense(self.w["embed"], self.final_state(h))


def argmax(x):
    """First index of the largest non-NaN value per row; -1 if every value is NaN."""
    x = np.asarray(x, dtype=np.float64)
    out = np.full(x.shape[0], -1, dtype=np.int64)
    for b in range(x.shape[0]):
        ok = ~np.isnan(x[b])
        if ok.any():
            m = np.max(x[b][ok])
            out[b] = int(np.flatnonzero(ok & (x[b] == m))[0])
    return out


def oda_step(model: Model, tokens, k_cache, v_cache, block_table, seq_lens, n_sink: int, window: int,
             score_fn, h_prev, tau: float, forced=None):
    """One ODA decode step on the decoder (Alg. 1): the Local forward (every
    restricted layer over S^L), the recall score q_t = R(h_{t-1}, E(x_t),
    h^L_t) from score_fn(h_prev, emb, h_local), the predicate (Full iff
    q_t > tau or nonfinite; a prescribed schedule replaces the comparison),
    the Full forward from the same pre-step history for flagged requests, and
    the selected state (App. A.5): its final hidden state, candidates, logits
    and greedy token.  The cache is not modified (oracle.step.commit does
    that).

    h^L_t is the final normalised Local hidden state (§2.1), and h_prev is the
    final normalised selected state of the previous step (App. A.5: the state
    the vocabulary projection reads); the result's "h_state" is that state
    for this step, the next step's h_prev."""
    from . import gate as Gt
    B = len(tokens)
    hL, kL, vL = model.forward(tokens, k_cache, v_cache, block_table, seq_lens,
                               lambda n: A.local_set(n, n_sink, window))
    emb = model.embed(tokens)
    hL_state = model.final_state(hL)
    score = score_fn(h_prev, emb, hL_state)
    flags = Gt.decide(score, tau, forced)
    work, n_work = Gt.compact(flags)
    h = hL.copy()
    kF = np.zeros_like(kL)
    vF = np.zeros_like(vL)
    if n_work:
        hF, kF_, vF_ = model.forward(tokens, k_cache, v_cache, block_table, seq_lens, A.full_set, requests=work)
        h[work] = hF[work]
        kF[:, work] = kF_[:, work]
        vF[:, work] = vF_[:, work]
    h_state = model.final_state(h)
    logits = dense(model.w["embed"], h_state)
    return dict(h_local=hL, h_local_state=hL_state, score=score, flags=flags.astype(np.int32), work_list=work,
                n_work=n_work, h=h, h_state=h_state, k_local=kL, v_local=vL, k_full=kF, v_full=vF, logits=logits,
                token=argmax(logits))
