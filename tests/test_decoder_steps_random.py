"""Seeded random whole ODA decode steps of the decoder around the hot path
(paper_2609_20734_amd.decoder) against the oracle's own steps: layer count,
widths, GQA group, head width, batch, lengths, Local sinks and window, head
kind and the prescribed Full schedule drawn per case; three steps each, the
oracle committing its own candidates, caches compared at the end (the
committed rows within a relative tolerance, everything else bit-exact).
Step tolerances as in test_decoder_parity.py."""
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
from test_decoder_parity import STEP_REL_L2, _rel_l2

pytestmark = pytest.mark.gpu


def _caches_close(got_k, got_v, ref_k, ref_v, table, seq0, T, L, Hkv):
    """Rows the steps committed (positions n0 - 1 .. n0 + T - 2 of every
    request, layer and KV head) within relative-L2 2e-3 of the oracle's (their
    inputs carry the hidden state's ~1e-4 difference, which can move elements
    near zero by many bf16 steps); every other element bit-exact."""
    gk, rk = OA.bf16_to_f64(got_k), OA.bf16_to_f64(ref_k)
    gv, rv = OA.bf16_to_f64(got_v), OA.bf16_to_f64(ref_v)
    written = np.zeros(gk.shape[:2] + (gk.shape[2], 16), dtype=bool)      # [L][NB][Hkv][slot]
    for b, n0 in enumerate(seq0):
        for p in range(int(n0) - 1, int(n0) - 1 + T):
            blk = table[b, p // 16]
            for l in range(L):
                for g in range(Hkv):
                    written[l, blk, g, p % 16] = True
                    for got, ref in ((gk[l, blk, g, :, p % 16, :].ravel(), rk[l, blk, g, :, p % 16, :].ravel()),
                                     (gv[l, blk, g, :, p % 16], rv[l, blk, g, :, p % 16])):
                        err = np.linalg.norm(got - ref)
                        assert err <= 2e-3 * np.linalg.norm(ref) + 1e-6, (b, p, l, g, err)
    wk = np.broadcast_to(written[:, :, :, None, :, None], gk.shape)
    wv = np.broadcast_to(written[:, :, :, None, :], gv.shape)
    assert np.array_equal(np.where(wk, 0, got_k), np.where(wk, 0, ref_k))
    assert np.array_equal(np.where(wv, 0, got_v), np.where(wv, 0, ref_v))


@pytest.mark.parametrize("seed", range(24))
def test_random_decoder_steps(seed):
    P = need_gpu()
    from paper_2609_20734_amd import decoder as PD
    g = np.random.default_rng(11000 + seed)
    L = int(g.integers(1, 4))
    d = 8 * int(g.integers(4, 33))
    Hkv = int(g.choice([1, 2]))
    Hq = Hkv * int(g.choice([1, 2, 4]))
    D = int(g.choice([64, 128]))
    F = 8 * int(g.integers(4, 49))
    V = 4 * int(g.integers(25, 250))
    B = int(g.integers(1, 5))
    T = 3
    seq0 = g.integers(1, 200, size=B).astype(np.int32)
    s = int(g.choice([0, 4]))
    W = int(g.integers(8, 80))
    head = str(g.choice(["paper", "mlp"]))
    dt = 4 * int(g.integers(2, 17))
    forced = (g.random((T, B)) < 0.5).astype(np.int32)

    shape = PD.DecoderShape(L, d, Hq, Hkv, D, F, V)
    w = S.decoder_weights(11000 + seed, L, d, Hq, Hkv, D, F, V)
    model = OD.Model(w, Hq, Hkv, D)
    mb = int(math.ceil((seq0.max() + T) / 16))
    table, nb = S.paged_block_table(S.rng(11000 + seed, S.STREAM_TABLE), seq0 + T, mb, permute=True)
    k, v = S.kv_cache(11000 + seed, L, nb, Hkv, D)
    gparams = S.gate_params(11000 + seed, head, d, dt)
    gate = P.gate_desc(P.HEAD_PAPER if head == "paper" else P.HEAD_MLP, d, dt, dev_f32(gparams), 1e-6)
    score_fn = (lambda hp, e, hl: OG.paper_head_score(gparams, d, dt, 1e-6, hp, e, hl)) if head == "paper" \
        else (lambda hp, e, hl: OG.mlp_score(gparams, d, dt, hl))
    tokens = S.tokens(11000 + seed, T, B, V)
    dw = {n: (dev_u16(a) if a.dtype == np.uint16 else dev_f32(a)) for n, a in w.items()}
    dk, dv, dtab, dseq = dev_u16(k), dev_u16(v), dev_i32(table), dev_i32(seq0)
    dec = PD.Decoder(shape, dw, B, dk, dv, dtab, dseq, mb, int(seq0.max()) + T, nb, s, W, gate=gate, tau=0.0,
                     prescribed=True)
    local, retry, out = dec.oda_stages()
    hk, hv, hseq = k.copy(), v.copy(), seq0.copy()
    h_prev = np.zeros((B, d))
    print(f"case {seed}: L={L} d={d} Hq={Hq} Hkv={Hkv} D={D} F={F} V={V} B={B} s={s} W={W} head={head} dt={dt}",
          flush=True)
    for step in range(T):
        dec.tokens.copy_(torch.from_numpy(tokens[step]))
        dec.forced.copy_(torch.from_numpy(forced[step]))
        for c in local + retry + out:
            c()
        torch.cuda.synchronize()
        r = OD.oda_step(model, tokens[step], hk, hv, table, hseq, s, W, score_fn, h_prev, 0.0, forced[step])
        np.testing.assert_array_equal(dec.flags.cpu().numpy(), forced[step])
        assert _rel_l2(dec.score.cpu().numpy(), r["score"]) <= STEP_REL_L2
        assert _rel_l2(dec.h.cpu().numpy(), r["h"]) <= STEP_REL_L2, f"step {step}: hidden"
        assert _rel_l2(dec.h_local.cpu().numpy(), r["h_local_state"]) <= STEP_REL_L2, f"step {step}: h^L_t"
        assert _rel_l2(dec.h_prev.cpu().numpy(), r["h_state"]) <= STEP_REL_L2, f"step {step}: h_t"
        assert _rel_l2(dec.logits.cpu().numpy(), r["logits"]) <= STEP_REL_L2, f"step {step}: logits"
        tok = dec.next_token.cpu().numpy()
        for b in range(B):
            top = np.sort(r["logits"][b])[-2:]
            if top[1] - top[0] > 1e-3 * max(1.0, abs(top[1])):
                assert tok[b] == r["token"][b], (step, b)
        OS.commit(hk, hv, table, hseq, r["k_local"], r["v_local"], r["k_full"], r["v_full"], forced[step])
        h_prev = r["h_state"]
        np.testing.assert_array_equal(dseq.cpu().numpy(), hseq)
    _caches_close(dk.cpu().numpy().view(np.uint16), dv.cpu().numpy().view(np.uint16), hk, hv, table, seq0, T, L,
                  Hkv)
    assert int(dec.counter.item()) == int(forced.sum())
