"""Direct-ring Local (App. A.5): per (layer, request, KV head) rings of whole
blocks holding the sinks and the recent window, filled from the paged cache
(oda_ring_fill), kept current by the commit (oda_commit_kv_ring) and read by
oda_local_decode_attn_ring with no block table.

* Filled from a cache, the ring call's out and lse equal the paged Local
  call's bit for bit (the same positions in the same order) and the fp64
  oracle's Local set within the bars; ring slots that hold no committed
  position are filled with NaN first and must not matter.  Cases: sinks 0 /
  4 / 20 (one and two sink blocks), windows inside and beyond the history,
  lengths 1 and 2 (nothing or one position committed), the candidate in
  k_cur or already in the ring, D = 64 / 128, GQA groups up to 16, forced
  splits, and a batch large enough that workgroups walk several layers.
* A growing-context loop of 100 steps with a 40-position window (the ring
  wraps every 80 positions): each step's ring Local equals the paged Local bit
  for bit, the commit writes the same candidate into both, and the final
  caches and lengths equal the oracle's replay of the commits.
"""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from harness import AttnProblem, check_close, dev_i32, dev_u16, need_gpu
from oracle import attention as OA
from oracle import step as OS

pytestmark = pytest.mark.gpu

NAN_BF16 = 0x7FC0


def _rings(P, shape, n_sink, window):
    n = P.ring_elements(shape, n_sink, window)
    kr = torch.full((n,), NAN_BF16, dtype=torch.int16, device="cuda")
    vr = torch.full((n,), NAN_BF16, dtype=torch.int16, device="cuda")
    return kr, vr


def _same_bits(a, b):
    return torch.equal(a.contiguous().view(torch.int32), b.contiguous().view(torch.int32))


@pytest.mark.parametrize("L,B,Hq,Hkv,D,seq,n_sink,window,split,cur", [
    (2, 3, 8, 2, 64, [1, 2, 40], 4, 16, 0, True),
    (1, 4, 16, 1, 128, [17, 300, 5, 1000], 4, 64, 2, True),
    (3, 2, 8, 8, 128, [515, 33], 20, 100, 0, False),
    (2, 2, 32, 8, 128, [70, 4000], 0, 2048, 6, True),
    (1, 3, 8, 4, 64, [16, 17, 32], 16, 16, 0, True),
    (2, 5, 4, 4, 64, [600, 1, 129, 128, 300], 4, 128, 4, False),
])
def test_ring_local_equals_paged_local(L, B, Hq, Hkv, D, seq, n_sink, window, split, cur):
    pb = AttnProblem(700 + L * 10 + B, L, B, Hq, Hkv, D, seq, cur=cur, split_blocks=split)
    P = pb.P
    kr, vr = _rings(P, pb.shape, n_sink, window)
    P.ring_fill(pb.shape, pb.dk, pb.dv, pb.dtable, pb.dseq, n_sink, window, kr, vr)
    paged = pb.run_local(n_sink, window)
    out, lse = pb.new_out(np.nan)
    ws = torch.zeros(max(256, P.attn_workspace_size(pb.shape, n_sink, window)), dtype=torch.uint8, device="cuda")
    ring_inp = P.inputs(pb.dq, None, None, None, pb.dseq, pb.scale, pb.dkc, pb.dvc)
    P.local_decode_attn_ring(pb.shape, ring_inp, kr, vr, n_sink, window, out, lse, ws)
    torch.cuda.synchronize()
    assert _same_bits(out, paged[0]) and _same_bits(lse, paged[1])
    want, want_lse, _ = pb.oracle_local(n_sink, window)
    check_close(out.cpu().numpy(), want, what="ring local")
    assert np.abs(lse.cpu().numpy() - want_lse).max() < 1e-4


def test_ring_local_in_the_layer_walk():
    """64 requests x 8 KV heads x 4 layers: the Local call's workgroups each
    walk all four layers of a (request, KV head), reading the ring."""
    seq = np.random.default_rng(71).integers(1, 300, size=64).tolist()
    pb = AttnProblem(71, 4, 64, 8, 8, 64, seq, cur=True)
    P = pb.P
    kr, vr = _rings(P, pb.shape, 4, 96)
    P.ring_fill(pb.shape, pb.dk, pb.dv, pb.dtable, pb.dseq, 4, 96, kr, vr)
    paged = pb.run_local(4, 96)
    out, lse = pb.new_out(np.nan)
    ws = torch.zeros(max(256, P.attn_workspace_size(pb.shape, 4, 96)), dtype=torch.uint8, device="cuda")
    P.local_decode_attn_ring(pb.shape, P.inputs(pb.dq, None, None, None, pb.dseq, pb.scale, pb.dkc, pb.dvc),
                             kr, vr, 4, 96, out, lse, ws)
    torch.cuda.synchronize()
    assert _same_bits(out, paged[0]) and _same_bits(lse, paged[1])


@pytest.mark.parametrize("D,G,n_sink", [(64, 4, 4), (128, 2, 20)])
def test_ring_decode_loop_with_commit(D, G, n_sink):
    P = need_gpu()
    L, B, Hkv, T = 2, 3, 2, 100
    Hq = Hkv * G
    W = 40
    seq0 = np.array([1, 30, 70], dtype=np.int32)
    mb = int(math.ceil((seq0.max() + T) / 16))
    table, nb = S.paged_block_table(S.rng(15, S.STREAM_TABLE), seq0 + T, mb, permute=True)
    k, v = S.kv_cache(15, L, nb, Hkv, D)
    q_all = S.normal_bf16(S.rng(16, S.STREAM_Q), (T, L, B, Hq, D))
    kc = S.normal_bf16(S.rng(17, S.STREAM_KCUR), (T, L, B, Hkv, D))
    vc = S.normal_bf16(S.rng(17, S.STREAM_VCUR), (T, L, B, Hkv, D))
    dk, dv, dtab, dseq = dev_u16(k), dev_u16(v), dev_i32(table), dev_i32(seq0)
    dq, dkc, dvc = (dev_u16(x) for x in (q_all, kc, vc))
    shape = P.Shape(L, B, Hq, Hkv, D, mb, int(seq0.max()) + T, nb, 0)
    kr, vr = _rings(P, shape, n_sink, W)
    P.ring_fill(shape, dk, dv, dtab, dseq, n_sink, W, kr, vr)
    ws_p = torch.zeros(max(256, P.attn_workspace_size(shape, n_sink, W)), dtype=torch.uint8, device="cuda")
    ws_r = torch.zeros_like(ws_p)
    ws_c = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    out_p, lse_p = (torch.empty(L, B, Hq, D, device="cuda"), torch.empty(L, B, Hq, device="cuda"))
    out_r, lse_r = torch.empty_like(out_p), torch.empty_like(lse_p)
    hk, hv, hseq = k.copy(), v.copy(), seq0.copy()
    scale = 1.0 / math.sqrt(D)
    for t in range(T):
        P.local_decode_attn(shape, P.inputs(dq[t], dk, dv, dtab, dseq, scale, dkc[t], dvc[t]), n_sink, W,
                            out_p, lse_p, ws_p)
        P.local_decode_attn_ring(shape, P.inputs(dq[t], None, None, None, dseq, scale, dkc[t], dvc[t]), kr, vr,
                                 n_sink, W, out_r, lse_r, ws_r)
        if t % 33 == 0 or t == T - 1:
            torch.cuda.synchronize()
            ref, _, _ = OA.decode_attention(q_all[t], hk, hv, table, hseq, lambda n: OA.local_set(n, n_sink, W),
                                            scale, k_cur=kc[t], v_cur=vc[t])
            check_close(out_r.cpu().numpy(), ref, what=f"ring step {t}")
        P.commit_kv_ring(shape, dk, dv, dtab, dseq, dkc[t], dvc[t], None, None, None, True, ws_c, kr, vr, n_sink, W)
        torch.cuda.synchronize()
        assert _same_bits(out_r, out_p) and _same_bits(lse_r, lse_p), f"step {t}"
        OS.commit(hk, hv, table, hseq, kc[t], vc[t], kc[t], vc[t], np.zeros(B, np.int32))
    assert np.array_equal(dseq.cpu().numpy(), hseq)
    assert np.array_equal(dk.cpu().numpy().view(np.uint16), hk) and np.array_equal(dv.cpu().numpy().view(np.uint16), hv)
