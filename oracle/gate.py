"""Recall gate, fp64, by definition.  TEST INFRASTRUCTURE (see package doc).

Two score functions:

* the recall head of App. A.2 (``paper_head_*``): three RMSNorm -> biased
  projection -> SiLU towers, the nine-part interaction vector, the fusion
  equation, two pre-RMSNorm residual SwiGLU blocks, a final RMSNorm and a
  biased scalar projection;
* a two-layer MLP stand-in d -> h -> 1 with exact-erf GELU (``mlp_*``).

Then the decision rule of §2.1 / Alg. 1: Full iff score > threshold or the
score is nonfinite, and the ascending list of flagged requests.
"""
from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------
# parameter packing (the C ABI's order; pinned by the parameter count)
# ---------------------------------------------------------------------------


def paper_head_shapes(d: int, dt: int):
    """Packed order of the App. A.2 head: per tower (h, e, l) the RMSNorm gain,
    the projection weight [dt][d] and its bias; the fusion weight [dt][9dt] and
    bias; per SwiGLU block the RMSNorm gain, gate [2dt][dt], up [2dt][dt] and
    down [dt][2dt] (bias-free); the final RMSNorm gain, w_o [dt] and b_o."""
    s = []
    for t in ("h", "e", "l"):
        s += [(f"rms_{t}", (d,)), (f"W_{t}", (dt, d)), (f"b_{t}", (dt,))]
    s += [("W_f", (dt, 9 * dt)), ("b_f", (dt,))]
    for k in (1, 2):
        s += [(f"rms_{k}", (dt,)), (f"W_gate_{k}", (2 * dt, dt)),
              (f"W_up_{k}", (2 * dt, dt)), (f"W_down_{k}", (dt, 2 * dt))]
    s += [("rms_o", (dt,)), ("w_o", (dt,)), ("b_o", (1,))]
    return s


def mlp_shapes(d: int, h: int):
    return [("W1", (h, d)), ("b1", (h,)), ("w2", (h,)), ("b2", (1,))]


def param_count(shapes) -> int:
    return int(sum(int(np.prod(shp)) for _, shp in shapes))


def unpack(params, shapes) -> dict:
    """Split a packed fp32 vector into named fp64 arrays."""
    params = np.asarray(params)
    assert params.size == param_count(shapes), (params.size, param_count(shapes))
    out, pos = {}, 0
    for name, shp in shapes:
        cnt = int(np.prod(shp))
        out[name] = params[pos:pos + cnt].astype(np.float64).reshape(shp)
        pos += cnt
    return out


# ---------------------------------------------------------------------------
# building blocks
# ---------------------------------------------------------------------------


def rmsnorm(x, w, eps: float):
    """RMSNorm with a gain and no bias: x / sqrt(mean(x^2) + eps) * w (row-wise)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def silu(x):
    """SiLU(x) = x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


_erf = np.vectorize(math.erf, otypes=[np.float64])


def gelu(x):
    """GELU with the exact error function: x * (1 + erf(x / sqrt 2)) / 2."""
    return 0.5 * x * (1.0 + _erf(np.asarray(x, dtype=np.float64) / math.sqrt(2.0)))


# ---------------------------------------------------------------------------
# scores
# ---------------------------------------------------------------------------


def paper_head_towers(p: dict, h_prev, emb, h_local, eps: float):
    """Tower outputs a, b, c for the inputs h_{t-1}, E(x_t), h_t^L (App. A.2)."""
    a = silu(rmsnorm(h_prev, p["rms_h"], eps) @ p["W_h"].T + p["b_h"])
    b = silu(rmsnorm(emb, p["rms_e"], eps) @ p["W_e"].T + p["b_e"])
    c = silu(rmsnorm(h_local, p["rms_l"], eps) @ p["W_l"].T + p["b_l"])
    return a, b, c


def interaction(a, b, c):
    """u = [a; b; c; a*b; |a-b|; a*c; |a-c|; b*c; |b-c|]  (App. A.2)."""
    return np.concatenate([a, b, c, a * b, np.abs(a - b), a * c, np.abs(a - c),
                           b * c, np.abs(b - c)], axis=-1)


def paper_head_score(params, d: int, dt: int, eps: float, h_prev, emb, h_local):
    """q_t = R_psi(h_{t-1}, E(x_t), h_t^L) of App. A.2 for a batch of rows."""
    p = unpack(params, paper_head_shapes(d, dt))
    a, b, c = paper_head_towers(p, h_prev, emb, h_local, eps)
    u = interaction(a, b, c)
    z = 0.5 * (a + b + c + silu(u @ p["W_f"].T + p["b_f"]))         # fusion equation
    for k in (1, 2):                                                # pre-norm residual SwiGLU
        r = rmsnorm(z, p[f"rms_{k}"], eps)
        z = z + (silu(r @ p[f"W_gate_{k}"].T) * (r @ p[f"W_up_{k}"].T)) @ p[f"W_down_{k}"].T
    return rmsnorm(z, p["rms_o"], eps) @ p["w_o"] + p["b_o"][0]


def mlp_score(params, d: int, h: int, x):
    """Stand-in logit w2 . GELU(W1 x + b1) + b2 (its sigmoid is the recall
    probability; the decision uses the logit)."""
    p = unpack(params, mlp_shapes(d, h))
    return gelu(np.asarray(x, dtype=np.float64) @ p["W1"].T + p["b1"]) @ p["w2"] + p["b2"][0]


# ---------------------------------------------------------------------------
# decision (§2.1, Alg. 1; App. A.5) and compaction
# ---------------------------------------------------------------------------


def decide(score, tau: float, forced=None) -> np.ndarray:
    """flag = 1 (Full) iff score > tau or score is nonfinite; with a prescribed
    schedule, flag = forced or nonfinite (App. B.7)."""
    score = np.asarray(score, dtype=np.float64)
    nonfinite = ~np.isfinite(score)
    if forced is not None:
        return (np.asarray(forced) != 0) | nonfinite
    return (score > tau) | nonfinite


def compact(flags):
    """Ascending indices of flagged requests and their count."""
    idx = np.flatnonzero(np.asarray(flags)).astype(np.int64)
    return idx, len(idx)
