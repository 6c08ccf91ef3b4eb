"""Whole-step HIP graph: a period of decode steps (Local -> gate -> Full ->
commit, per step) captured once and replayed, against the same steps run
eagerly from the same state and against the fp64 oracle's replay of the
period (its own attention, selection and commit on host copies).  Replays are
separated by eager work and host synchronisation, and every replay is checked:
each step's outputs against the oracle within the attention bar, and outputs,
final caches, lengths and recall counter bit-identical to the eager run (the
caches and lengths also equal the oracle's bit for bit).  One case reads
Local from direct-ring rings that the captured commits keep current."""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from harness import LSE_ABS, check_close, dev_f32, dev_i32, dev_u16, need_gpu
from oracle import attention as OA
from oracle import step as OS

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt,local", [(16, "paged"), (64, "paged"), (16, "ring")])   # two tower widths; Local
def test_graph_replay_matches_eager(dt, local):                                      # from the cache or the rings
    P = need_gpu()
    L, B, Hkv, G, D, T = 2, 3, 2, 4, 128, 8
    Hq = Hkv * G
    s, W = 4, 24
    seq0 = np.array([9, 40, 100], dtype=np.int32)
    mb = int(math.ceil((seq0.max() + 4 * T) / 16))
    table, nb = S.paged_block_table(S.rng(1, S.STREAM_TABLE), seq0 + 4 * T, mb)
    k, v = S.kv_cache(1, L, nb, Hkv, D)
    q = dev_u16(S.normal_bf16(S.rng(2, S.STREAM_Q), (T, L, B, Hq, D)))
    kl, vl, kf, vf = (dev_u16(S.normal_bf16(S.rng(3 + i, S.STREAM_KCUR), (T, L, B, Hkv, D))) for i in range(4))
    sched = np.stack([S.periodic_schedule(T, 2)] * B, axis=1).astype(np.int32)   # first 2 of every T -> Full
    forced = dev_i32(sched)
    d = 64
    gate = P.gate_desc(P.HEAD_PAPER, d, dt, dev_f32(S.gate_params(4, "paper", d, dt)))
    h, e, hl = (dev_f32(x) for x in S.gate_inputs(4, T, B, d))
    q_h = S.normal_bf16(S.rng(2, S.STREAM_Q), (T, L, B, Hq, D))
    cand_h = [S.normal_bf16(S.rng(3 + i, S.STREAM_KCUR), (T, L, B, Hkv, D)) for i in range(4)]
    shape = P.Shape(L, B, Hq, Hkv, D, mb, int(seq0.max()) + 4 * T, nb, 4)
    k0, v0 = dev_u16(k), dev_u16(v)
    dk, dv = k0.clone(), v0.clone()
    dtab = dev_i32(table)
    seq_init = dev_i32(seq0)
    dseq = seq_init.clone()
    ws_l = torch.zeros(max(256, P.attn_workspace_size(shape, s, W)), dtype=torch.uint8, device="cuda")
    ws_f = torch.zeros(max(256, P.attn_workspace_size(shape, 0, 0)), dtype=torch.uint8, device="cuda")
    ws_g = torch.zeros(P.gate_workspace_size(gate, B), dtype=torch.uint8, device="cuda")
    ws_c = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    score = torch.empty(B, device="cuda")
    flags = torch.empty(B, dtype=torch.int32, device="cuda")
    wl = torch.empty(B, dtype=torch.int32, device="cuda")
    nw = torch.empty(1, dtype=torch.int32, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int64, device="cuda")
    outs = torch.zeros(T, L, B, Hq, D, device="cuda")
    lses = torch.zeros(T, L, B, Hq, device="cuda")
    scale = 1.0 / math.sqrt(D)

    ring = local == "ring"
    if ring:   # direct-ring Local: rings refilled from the cache at every reset, kept current by the commit
        n_ring = P.ring_elements(shape, s, W)
        kr = torch.full((n_ring,), 0x7FC0, dtype=torch.int16, device="cuda")
        vr = torch.full((n_ring,), 0x7FC0, dtype=torch.int16, device="cuda")

    def period():
        for t in range(T):
            if ring:
                P.local_decode_attn_ring(shape, P.inputs(q[t], None, None, None, dseq, scale, kl[t], vl[t]), kr, vr,
                                         s, W, outs[t], lses[t], ws_l)
            else:
                P.local_decode_attn(shape, P.inputs(q[t], dk, dv, dtab, dseq, scale, kl[t], vl[t]), s, W, outs[t],
                                    lses[t], ws_l)
            P.recall_gate(gate, B, h[t], e[t], hl[t], 0.0, forced[t], score, flags, wl, nw, ctr, ws_g)
            P.full_decode_attn(shape, P.inputs(q[t], dk, dv, dtab, dseq, scale, kf[t], vf[t]), 0, None, wl, nw,
                               outs[t], lses[t], ws_f)
            if ring:
                P.commit_kv_ring(shape, dk, dv, dtab, dseq, kl[t], vl[t], kf[t], vf[t], flags, True, ws_c,
                                 k_ring=kr, v_ring=vr, n_sink=s, window=W)
            else:
                P.commit_kv(shape, dk, dv, dtab, dseq, kl[t], vl[t], kf[t], vf[t], flags, True, ws_c)

    def reset():
        dk.copy_(k0)
        dv.copy_(v0)
        dseq.copy_(seq_init)
        if ring:
            P.ring_fill(shape, dk, dv, dtab, dseq, s, W, kr, vr)
        ctr.zero_()
        outs.zero_()
        lses.zero_()

    # the oracle's replay of the period: Local with the Local candidate, Full
    # with the Full candidate for the scheduled requests, the selected rows,
    # then the commit of the selected candidates
    hk, hv, hseq = k.copy(), v.copy(), seq0.copy()
    want = []
    for t in range(T):
        loc = OA.decode_attention(q_h[t], hk, hv, table, hseq, lambda n: OA.local_set(n, s, W), scale,
                                  k_cur=cand_h[0][t], v_cur=cand_h[1][t])
        full = OA.decode_attention(q_h[t], hk, hv, table, hseq, OA.full_set, scale, k_cur=cand_h[2][t],
                                   v_cur=cand_h[3][t])
        o, l_ = loc[0].copy(), loc[1].copy()
        for b in np.flatnonzero(sched[t]):
            o[:, b], l_[:, b] = full[0][:, b], full[1][:, b]
        want.append((o, l_))
        OS.commit(hk, hv, table, hseq, cand_h[0][t], cand_h[1][t], cand_h[2][t], cand_h[3][t], sched[t])

    def check_against_oracle(tag):
        o_all, l_all = outs.cpu().numpy(), lses.cpu().numpy()
        for t in range(T):
            check_close(o_all[t], want[t][0], what=f"{tag} step {t}")
            assert np.max(np.abs(l_all[t] - want[t][1])) <= LSE_ABS
        assert np.array_equal(dk.cpu().numpy().view(np.uint16), hk)
        assert np.array_equal(dv.cpu().numpy().view(np.uint16), hv)
        assert dseq.cpu().numpy().tolist() == hseq.tolist()
        assert int(ctr.item()) == int(sched.sum())

    reset()
    period()                     # eager reference (also warms up every kernel)
    torch.cuda.synchronize()
    check_against_oracle("eager")
    ref = [x.clone() for x in (outs, lses, dk, dv, dseq, ctr)]
    assert int(ctr.item()) == 2 * B

    g = torch.cuda.CUDAGraph()
    reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        period()
    for rep in range(3):
        reset()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (outs, lses, dk, dv, dseq, ctr)
        for a, b_ in zip(got, ref):
            assert torch.equal(a, b_), f"replay {rep} differs from eager"
        check_against_oracle(f"replay {rep}")
        _ = (outs * 2).sum().item()          # unrelated eager work between replays
