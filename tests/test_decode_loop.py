"""A growing-context ODA decode loop on the GPU (Alg. 1 with the commit of
App. A.5): every step runs Local with the Local candidate, the gate under a
prescribed schedule, Full with the Full candidate for flagged requests, and
oda_commit_kv of the selected candidate.  The fp64 oracle replays the same
steps on host copies; outputs match at every step and the final caches match
bit for bit."""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from harness import check_close, dev_f32, dev_i32, dev_u16, need_gpu
from oracle import attention as OA
from oracle import step as OS

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("D,G", [(128, 4), (64, 8)])
def test_decode_loop_with_commit(D, G):
    P = need_gpu()
    L, B, Hkv, T = 2, 3, 2, 12
    Hq = Hkv * G
    s, W = 4, 24
    seq0 = np.array([1, 30, 70], dtype=np.int32)       # the first candidate sits at n - 1
    mb = int(math.ceil((seq0.max() + T) / 16))
    table, nb = S.paged_block_table(S.rng(5, S.STREAM_TABLE), seq0 + T, mb, permute=True)
    k, v = S.kv_cache(5, L, nb, Hkv, D)
    q_all = S.normal_bf16(S.rng(6, S.STREAM_Q), (T, L, B, Hq, D))
    kl = S.normal_bf16(S.rng(7, S.STREAM_KCUR), (T, L, B, Hkv, D))
    vl = S.normal_bf16(S.rng(7, S.STREAM_VCUR), (T, L, B, Hkv, D))
    kf = S.normal_bf16(S.rng(8, S.STREAM_KCUR), (T, L, B, Hkv, D))
    vf = S.normal_bf16(S.rng(8, S.STREAM_VCUR), (T, L, B, Hkv, D))
    forced = (S.rng(9, S.STREAM_FORCED).random((T, B)) < 0.4).astype(np.int32)
    d = 64
    params = S.gate_params(3, "mlp", d, 16)
    h, e, hl = S.gate_inputs(3, T, B, d)

    dk, dv, dtab, dseq = dev_u16(k), dev_u16(v), dev_i32(table), dev_i32(seq0)
    dq, dkl, dvl, dkf, dvf = (dev_u16(x) for x in (q_all, kl, vl, kf, vf))
    dforced = dev_i32(forced)
    gate = P.gate_desc(P.HEAD_MLP, d, 16, dev_f32(params))
    dh, de, dhl = dev_f32(h), dev_f32(e), dev_f32(hl)
    shape = P.Shape(L, B, Hq, Hkv, D, mb, int(seq0.max()) + T, nb, 2)
    ws_l = torch.zeros(max(1, P.attn_workspace_size(shape, s, W)), dtype=torch.uint8, device="cuda")
    ws_f = torch.zeros(max(1, P.attn_workspace_size(shape, 0, 0)), dtype=torch.uint8, device="cuda")
    ws_g = torch.zeros(P.gate_workspace_size(gate, B), dtype=torch.uint8, device="cuda")
    ws_c = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    score = torch.empty(B, device="cuda")
    flags = torch.empty(B, dtype=torch.int32, device="cuda")
    wl = torch.empty(B, dtype=torch.int32, device="cuda")
    nw = torch.empty(1, dtype=torch.int32, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int64, device="cuda")
    out = torch.empty(L, B, Hq, D, device="cuda")
    lse = torch.empty(L, B, Hq, device="cuda")

    hk, hv, hseq = k.copy(), v.copy(), seq0.copy()
    scale = 1.0 / math.sqrt(D)
    for t in range(T):
        inp_l = P.inputs(dq[t], dk, dv, dtab, dseq, scale, dkl[t], dvl[t])
        inp_f = P.inputs(dq[t], dk, dv, dtab, dseq, scale, dkf[t], dvf[t])
        P.local_decode_attn(shape, inp_l, s, W, out, lse, ws_l)
        P.recall_gate(gate, B, dh[t], de[t], dhl[t], 0.0, dforced[t], score, flags, wl, nw, ctr, ws_g)
        P.full_decode_attn(shape, inp_f, 0, None, wl, nw, out, lse, ws_f)
        P.commit_kv(shape, dk, dv, dtab, dseq, dkl[t], dvl[t], dkf[t], dvf[t], flags, True, ws_c)
        torch.cuda.synchronize()

        ref_l = OA.decode_attention(q_all[t], hk, hv, table, hseq, lambda n: OA.local_set(n, s, W), scale,
                                    k_cur=kl[t], v_cur=vl[t])
        ref_f = OA.decode_attention(q_all[t], hk, hv, table, hseq, OA.full_set, scale, k_cur=kf[t], v_cur=vf[t])
        sel = forced[t].astype(bool)
        ref = np.where(sel[None, :, None, None], ref_f[0], ref_l[0])
        assert np.array_equal(flags.cpu().numpy(), forced[t])
        check_close(out.cpu().numpy(), ref, what=f"step {t}")
        OS.commit(hk, hv, table, hseq, kl[t], vl[t], kf[t], vf[t], forced[t])
        assert np.array_equal(dseq.cpu().numpy(), hseq)

    assert int(ctr.item()) == int(forced.sum())
    assert np.array_equal(dk.cpu().numpy().view(np.uint16), hk)
    assert np.array_equal(dv.cpu().numpy().view(np.uint16), hv)
