"""GPU parity of the decoder around the hot path (oda_dense_bf16,
oda_qk_norm_rope, oda_embed_bf16, oda_copy_rows, oda_argmax) and of whole ODA
decode steps composed from them (paper_2609_20734_amd.decoder), against the
fp64 oracle (oracle/decoder.py).

Tolerances.  Dense layers: fp32 accumulation of bf16 x fp32 products over K
<= 6,144 terms, |err| <= 1e-4 of the output scale.  q/k/v candidates are
rounded to bf16 by both sides from fp32 (GPU) and fp64 (oracle) values, so an
element within ~1e-7 of a rounding boundary may land one bf16 step apart:
such elements must be rare (< 0.5%) and exactly one step off.  Whole steps:
those rare one-step differences move the hidden state by ~1e-4 of its scale;
hidden states and logits are held to relative-L2 1e-3, and the greedy token
must agree unless the oracle's top two logits are within 1e-3 of each other.
"""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from harness import dev_f32, dev_i32, dev_u16, need_gpu
from oracle import attention as OA
from oracle import decoder as OD
from oracle import gate as OG
from oracle import step as OS

pytestmark = pytest.mark.gpu

DENSE_REL = 1e-4
STEP_REL_L2 = 1e-3


def _bf16_close(got_bits, ref_bits, what):
    """Equal except for rare elements exactly one bf16 step apart."""
    g = np.asarray(got_bits, dtype=np.uint16).view(np.int16).astype(np.int64)
    r = np.asarray(ref_bits, dtype=np.uint16).view(np.int16).astype(np.int64)
    gv, rv = OA.bf16_to_f64(got_bits), OA.bf16_to_f64(ref_bits)
    diff = gv != rv
    if diff.any():
        assert diff.mean() < 5e-3, f"{what}: {diff.mean():.2%} of elements differ"
        assert np.all(np.abs(g[diff] - r[diff]) == 1) and np.all(np.sign(gv[diff]) == np.sign(rv[diff])), \
            f"{what}: a difference larger than one bf16 step"


def _rel_l2(got, ref):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


@pytest.mark.parametrize("K,N,B,mode,norm,res,listed", [
    (64, 5, 1, "plain", False, False, False),
    (72, 96, 3, "plain", True, True, False),        # ragged chunk tail, norm + residual
    (512, 40, 9, "plain", True, False, True),       # two batch tiles, a selection list
    (1040, 33, 2, "swiglu", True, False, False),
    (2048, 64, 5, "swiglu", True, False, True),
    (6144, 24, 1, "plain", False, True, False),     # the Qwen3-1.7B down projection's K
])
def test_dense(K, N, B, mode, norm, res, listed):
    P = need_gpu()
    g = S.rng(K + N + B, S.STREAM_DECODER)
    rows = 2 * N if mode == "swiglu" else N
    W = S.normal_bf16(g, (rows, K), K ** -0.5)
    x = g.standard_normal((B, K)).astype(np.float32)
    gain = (1 + 0.02 * g.standard_normal(K)).astype(np.float32) if norm else None
    r = g.standard_normal((B, N)).astype(np.float32) if res else None
    sel = [b for b in range(B) if b % 2 == 0][::-1] if listed else list(range(B))
    desc = P.dense_desc(K, N, P.DENSE_SWIGLU if mode == "swiglu" else P.DENSE_PLAIN, dev_u16(W),
                        dev_f32(gain) if norm else None, 1e-6)
    y = torch.full((B, N), 7.0, device="cuda")
    wl = dev_i32(sel + [0] * (B - len(sel))) if listed else None
    nw = dev_i32([len(sel)]) if listed else None
    P.dense_bf16(desc, B, dev_f32(x), dev_f32(r) if res else None, y, wl, nw)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    if mode == "swiglu":
        ref = OD.swiglu(W, x[sel], gain, 1e-6)
    else:
        ref = OD.dense(W, x[sel], gain, 1e-6, r[sel] if res else None)
    scale = max(1.0, float(np.abs(ref).max()))
    assert np.abs(got[sel] - ref).max() <= DENSE_REL * scale
    others = [b for b in range(B) if b not in sel]
    assert np.all(got[others] == 7.0)


def test_dense_residual_in_place():
    P = need_gpu()
    g = S.rng(5, S.STREAM_DECODER)
    W = S.normal_bf16(g, (48, 256), 256 ** -0.5)
    x = g.standard_normal((3, 256)).astype(np.float32)
    h = g.standard_normal((3, 48)).astype(np.float32)
    dh = dev_f32(h)
    P.dense_bf16(P.dense_desc(256, 48, P.DENSE_PLAIN, dev_u16(W)), 3, dev_f32(x), dh, dh)
    torch.cuda.synchronize()
    ref = OD.dense(W, x, residual=h)
    assert np.abs(dh.cpu().numpy() - ref).max() <= DENSE_REL * max(1.0, float(np.abs(ref).max()))


@pytest.mark.parametrize("D,Hq,Hkv,gains,listed", [(128, 16, 8, True, False), (64, 8, 2, False, True),
                                                    (128, 4, 4, True, True)])
def test_qk_norm_rope(D, Hq, Hkv, gains, listed):
    P = need_gpu()
    B = 4
    g = S.rng(D + Hq, S.STREAM_DECODER)
    qkv = (3 * g.standard_normal((B, (Hq + 2 * Hkv) * D))).astype(np.float32)
    qg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32) if gains else None
    kg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32) if gains else None
    seq = np.array([1, 17, 131072, 516788], dtype=np.int32)      # positions 0 ... 516,787
    sel = [3, 0, 2] if listed else list(range(B))
    q = torch.full((B, Hq, D), 5.0, dtype=torch.bfloat16, device="cuda")
    k = torch.full((B, Hkv, D), 5.0, dtype=torch.bfloat16, device="cuda")
    v = torch.full((B, Hkv, D), 5.0, dtype=torch.bfloat16, device="cuda")
    wl = dev_i32(sel + [0] * (B - len(sel))) if listed else None
    nw = dev_i32([len(sel)]) if listed else None
    P.qk_norm_rope(B, Hq, Hkv, D, dev_f32(qkv), dev_f32(qg) if gains else None, dev_f32(kg) if gains else None,
                   1e-6, 1e6, dev_i32(seq), q, k, v, wl, nw)
    torch.cuda.synchronize()
    rq, rk, rv = OD.qk_norm_rope(qkv[sel], Hq, Hkv, D, qg, kg, 1e-6, 1e6, seq[sel] - 1)
    bits = lambda t: t.cpu().view(torch.int16).numpy().view(np.uint16)
    _bf16_close(bits(q)[sel], OD.bf16_bits(rq), "q")
    _bf16_close(bits(k)[sel], OD.bf16_bits(rk), "k")
    np.testing.assert_array_equal(bits(v)[sel], OD.bf16_bits(rv))        # v: one rounding of the input
    others = [b for b in range(B) if b not in sel]
    assert torch.all(q.cpu()[others] == 5.0)


def test_embed_copy_rows_argmax():
    P = need_gpu()
    g = S.rng(11, S.STREAM_DECODER)
    V, d, B = 1000, 64, 4
    table = S.normal_bf16(g, (V, d))
    toks = np.array([0, 999, 17, 1000], dtype=np.int32)          # the last one is out of range
    x = torch.zeros(B, d, device="cuda")
    P.embed_bf16(dev_u16(table), V, d, B, dev_i32(toks), x)
    torch.cuda.synchronize()
    got = x.cpu().numpy()
    np.testing.assert_array_equal(got[:3], OA.bf16_to_f64(table[toks[:3]]))
    assert np.isnan(got[3]).all()

    src = g.standard_normal((B, 8)).astype(np.float32)
    dst = torch.full((B, 8), -1.0, device="cuda")
    P.copy_rows(B, 8, dev_f32(src), dst, dev_i32([2, 0, 0, 0]), dev_i32([2]))
    torch.cuda.synchronize()
    out = dst.cpu().numpy()
    np.testing.assert_array_equal(out[[0, 2]], src[[0, 2]])
    assert np.all(out[[1, 3]] == -1.0)

    n = 151936
    logits = g.standard_normal((3, n)).astype(np.float32)
    logits[1, 5] = logits[1, 70000] = 50.0                          # a tie: the first index wins
    logits[2] = np.nan
    logits[2, n - 1] = -3.0
    idx = torch.zeros(3, dtype=torch.int32, device="cuda")
    P.argmax(3, n, dev_f32(logits), idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(idx.cpu().numpy(), OD.argmax(logits))
    assert idx.cpu().numpy()[1] == 5 and idx.cpu().numpy()[2] == n - 1


class Tiny:
    """A 2-layer decoder over a paged cache, on the device and in the oracle."""

    def __init__(self, seed=3, B=3, T=4, seq0=(1, 30, 90), s=4, W=24, head="paper", fused_prep=True):
        P = self.P = need_gpu()
        from paper_2609_20734_amd import decoder as PD
        L, d, Hq, Hkv, D, F, V = 2, 128, 4, 2, 64, 192, 512
        self.shape = PD.DecoderShape(L, d, Hq, Hkv, D, F, V)
        self.w = S.decoder_weights(seed, L, d, Hq, Hkv, D, F, V)
        self.model = OD.Model(self.w, Hq, Hkv, D)
        self.seq0 = np.array(seq0, dtype=np.int32)
        self.mb = int(math.ceil((self.seq0.max() + T) / 16))
        self.table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), self.seq0 + T, self.mb, permute=True)
        self.k, self.v = S.kv_cache(seed, L, nb, Hkv, D)
        self.s, self.W, self.B, self.T = s, W, B, T
        dt = 32
        self.gparams = S.gate_params(seed, head, d, dt)
        kind = P.HEAD_PAPER if head == "paper" else P.HEAD_MLP
        self.gate = P.gate_desc(kind, d, dt, dev_f32(self.gparams), 1e-6)
        self.score_fn = (lambda hp, e, hl: OG.paper_head_score(self.gparams, d, dt, 1e-6, hp, e, hl)) \
            if head == "paper" else (lambda hp, e, hl: OG.mlp_score(self.gparams, d, dt, hl))
        self.tokens = S.tokens(seed, T, B, V)
        dw = {n: (dev_u16(a) if a.dtype == np.uint16 else dev_f32(a)) for n, a in self.w.items()}
        self.dk, self.dv = dev_u16(self.k), dev_u16(self.v)
        self.dtab, self.dseq = dev_i32(self.table), dev_i32(self.seq0)
        self.dec = PD.Decoder(self.shape, dw, B, self.dk, self.dv, self.dtab, self.dseq, self.mb,
                              int(self.seq0.max()) + T, nb, s, W, gate=self.gate, tau=0.0, prescribed=True,
                              fused_prep=fused_prep)


def test_decoder_steps_match_oracle():
    """Four ODA steps with prescribed flags (some steps without any Full
    retry, some with all requests), each checked against the oracle's own
    step; the oracle commits its own candidates, so the histories of the two
    sides evolve independently and are compared at the end."""
    t = Tiny()
    P, dec = t.P, t.dec
    forced = np.array([[0, 1, 0], [0, 0, 0], [1, 1, 1], [1, 0, 1]], dtype=np.int32)
    local, retry, out = dec.oda_stages()
    hk, hv, hseq = t.k.copy(), t.v.copy(), t.seq0.copy()
    h_prev = np.zeros((t.B, t.shape.d_model))
    for step in range(t.T):
        dec.tokens.copy_(torch.from_numpy(t.tokens[step]))
        dec.forced.copy_(torch.from_numpy(forced[step]))
        for c in local + retry + out:
            c()
        torch.cuda.synchronize()
        r = OD.oda_step(t.model, t.tokens[step], hk, hv, t.table, hseq, t.s, t.W, t.score_fn, h_prev, 0.0,
                        forced[step])
        np.testing.assert_array_equal(dec.flags.cpu().numpy(), forced[step])
        assert int(dec.n_work.item()) == int(forced[step].sum())
        assert _rel_l2(dec.score.cpu().numpy(), r["score"]) <= STEP_REL_L2
        assert _rel_l2(dec.h.cpu().numpy(), r["h"]) <= STEP_REL_L2, f"step {step}: hidden"
        # the head's inputs: final-normalised Local state and the carried selected state
        assert _rel_l2(dec.h_local.cpu().numpy(), r["h_local_state"]) <= STEP_REL_L2, f"step {step}: h^L_t"
        assert _rel_l2(dec.h_prev.cpu().numpy(), r["h_state"]) <= STEP_REL_L2, f"step {step}: h_t"
        assert _rel_l2(dec.logits.cpu().numpy(), r["logits"]) <= STEP_REL_L2, f"step {step}: logits"
        tok = dec.next_token.cpu().numpy()
        for b in range(t.B):
            top = np.sort(r["logits"][b])[-2:]
            if top[1] - top[0] > 1e-3 * max(1.0, abs(top[1])):
                assert tok[b] == r["token"][b], (step, b)
        for name in ("k_local", "v_local"):
            got = getattr(dec, "k_loc" if name == "k_local" else "v_loc").cpu().view(torch.int16).numpy()
            _bf16_close(got.view(np.uint16), r[name], f"step {step} {name}")
        OS.commit(hk, hv, t.table, hseq, r["k_local"], r["v_local"], r["k_full"], r["v_full"], forced[step])
        h_prev = r["h_state"]
        np.testing.assert_array_equal(t.dseq.cpu().numpy(), hseq)
    _bf16_close(t.dk.cpu().numpy().view(np.uint16), hk, "K cache")
    _bf16_close(t.dv.cpu().numpy().view(np.uint16), hv, "V cache")
    assert int(dec.counter.item()) == int(forced.sum())


def test_fused_preparation_steps_equal_separate_launches():
    """Whole ODA steps with each attention call preparing its own query and
    candidate (oda_*_decode_attn_qkv) equal, bit for bit, the same steps with
    oda_qk_norm_rope as a launch of its own: hidden states, scores, logits,
    tokens, caches and lengths."""
    forced = np.array([[1, 0, 1], [0, 0, 0], [1, 1, 1], [0, 1, 0]], dtype=np.int32)
    results = []
    for fused in (True, False):
        t = Tiny(seed=6, fused_prep=fused)
        dec = t.dec
        local, retry, out = dec.oda_stages()
        per_step = []
        for step in range(t.T):
            dec.tokens.copy_(torch.from_numpy(t.tokens[step]))
            dec.forced.copy_(torch.from_numpy(forced[step]))
            for c in local + retry + out:
                c()
            torch.cuda.synchronize()
            per_step.append([x.clone() for x in (dec.h, dec.h_prev, dec.score, dec.logits, dec.next_token)])
        results.append((per_step, t.dk.clone(), t.dv.clone(), t.dseq.clone()))
    (fa, fk, fv, fs), (ua, uk, uv, us) = results
    for step, (a, b) in enumerate(zip(fa, ua)):
        for x, y in zip(a, b):
            assert torch.equal(x, y), step
    assert torch.equal(fk, uk) and torch.equal(fv, uv) and torch.equal(fs, us)


def test_decoder_stage_graphs_replay_bit_exactly():
    """The three stages of a step captured as HIP graphs (no memset nodes)
    and replayed three times, with a reset, unrelated eager work and host
    synchronisation between replays, give the eager run's results bit for bit."""
    t = Tiny(seed=4, head="mlp")
    dec = t.dec
    forced = np.array([1, 0, 1], dtype=np.int32)
    stages = dec.oda_stages()
    k0, v0 = t.dk.clone(), t.dv.clone()

    def reset():
        t.dk.copy_(k0)
        t.dv.copy_(v0)
        t.dseq.copy_(torch.from_numpy(t.seq0))
        dec.counter.zero_()
        dec.h_prev.zero_()
        dec.tokens.copy_(torch.from_numpy(t.tokens[0]))
        dec.forced.copy_(torch.from_numpy(forced))

    def outputs():
        return [x.clone() for x in (dec.logits, dec.next_token, dec.h_prev, t.dk, t.dv, t.dseq, dec.counter)]

    reset()
    for st in stages:
        for c in st:
            c()
    torch.cuda.synchronize()
    ref = outputs()
    graphs = []
    reset()
    torch.cuda.synchronize()
    for i in range(len(stages)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            # prepared calls bind the current stream: prepare them on the capture stream
            for c in dec.oda_stages()[i]:
                c()
        graphs.append(g)
    for rep in range(3):
        reset()
        torch.cuda.synchronize()
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outputs(), ref):
            assert torch.equal(a, b), f"replay {rep} differs from eager"
        _ = (dec.logits * 2).sum().item()
