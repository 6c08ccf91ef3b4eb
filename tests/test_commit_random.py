"""Seeded random selected-state commits (App. A.5 commit equation) against
the oracle's commit: layer count, batch, KV heads, head width, lengths
(block boundaries included), per-request flags, with and without the Full
candidates, the length advance on or off, dense or padded layer strides;
half the cases also keep direct-ring Local rings current, checked by a Local
call at the new lengths against the paged one (bit for bit)."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import dev_i32, dev_u16, need_gpu
from oracle import step as OS

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(30))
def test_random_commits(seed):
    P = need_gpu()
    g = np.random.default_rng(6000 + seed)
    L = int(g.integers(1, 5))
    B = int(g.integers(1, 11))
    Hkv = int(g.choice([1, 2, 4, 8]))
    D = int(g.choice([64, 128]))
    seq = g.choice([1, 15, 16, 17, 31, 32, 33, int(g.integers(1, 300))], size=B).astype(np.int32)
    with_full = bool(g.random() < 0.7)
    advance = bool(g.random() < 0.8)
    flags = (g.random(B) < 0.5).astype(np.int32)
    mb = int(np.ceil((seq.max() + 1) / 16))   # room for a Local call at the advanced lengths
    table, nb = S.paged_block_table(S.rng(6000 + seed, S.STREAM_TABLE), seq, mb, permute=True, extra_blocks=2)
    k, v = S.kv_cache(6000 + seed, L, nb, Hkv, D)
    kl = S.normal_bf16(S.rng(6100 + seed, S.STREAM_KCUR), (L, B, Hkv, D))
    vl = S.normal_bf16(S.rng(6100 + seed, S.STREAM_VCUR), (L, B, Hkv, D))
    kf = S.normal_bf16(S.rng(6200 + seed, S.STREAM_KCUR), (L, B, Hkv, D))
    vf = S.normal_bf16(S.rng(6200 + seed, S.STREAM_VCUR), (L, B, Hkv, D))
    dense = nb * Hkv * 16 * D
    stride = dense + 8 * int(g.integers(1, 50)) if g.random() < 0.5 else 0
    if stride:
        dk = torch.zeros(L * stride, dtype=torch.int16, device="cuda")
        dv = torch.zeros(L * stride, dtype=torch.int16, device="cuda")
        for l in range(L):
            dk[l * stride:l * stride + dense] = torch.from_numpy(k[l].reshape(-1).view(np.int16)).cuda()
            dv[l * stride:l * stride + dense] = torch.from_numpy(v[l].reshape(-1).view(np.int16)).cuda()
    else:
        dk, dv = dev_u16(k), dev_u16(v)
    dseq = dev_i32(seq)
    dtable = dev_i32(table)
    shape = P.Shape(L, B, Hkv, Hkv, D, mb, int(seq.max()), nb, layer_stride_kv=stride)
    ws = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    # half the cases commit into direct-ring Local rings too (filled at the pre-commit lengths)
    ring = bool(g.random() < 0.5)
    n_sink, window = int(g.choice([0, 4, 20])), int(g.integers(16, 200))
    args = (shape, dk, dv, dtable, dseq, dev_u16(kl), dev_u16(vl), dev_u16(kf) if with_full else None,
            dev_u16(vf) if with_full else None, dev_i32(flags) if with_full else None, advance, ws)
    if ring:
        n = P.ring_elements(shape, n_sink, window)
        kr = torch.full((n,), 0x7FC0, dtype=torch.int16, device="cuda")
        vr = torch.full((n,), 0x7FC0, dtype=torch.int16, device="cuda")
        P.ring_fill(shape, dk, dv, dtable, dseq, n_sink, window, kr, vr)
        P.commit_kv_ring(*args, k_ring=kr, v_ring=vr, n_sink=n_sink, window=window)
    else:
        P.commit_kv(*args)
    torch.cuda.synchronize()
    hk, hv, hseq = k.copy(), v.copy(), seq.copy()
    sel = flags if with_full else np.zeros(B, np.int32)
    OS.commit(hk, hv, table, hseq, kl, vl, kf if with_full else kl, vf if with_full else vl, sel)
    if stride:
        gk = np.stack([dk[l * stride:l * stride + dense].cpu().numpy() for l in range(L)]).reshape(k.shape)
        gv = np.stack([dv[l * stride:l * stride + dense].cpu().numpy() for l in range(L)]).reshape(v.shape)
        assert not dk.view(L, stride)[:, dense:].any() and not dv.view(L, stride)[:, dense:].any()  # padding untouched
    else:
        gk, gv = dk.cpu().numpy(), dv.cpu().numpy()
    assert np.array_equal(gk.view(np.uint16), hk)
    assert np.array_equal(gv.view(np.uint16), hv)
    assert dseq.cpu().numpy().tolist() == (hseq if advance else seq).tolist()
    assert int(ws.sum().item()) == 0      # the tickets are back at zero
    if ring:
        # Local at the new lengths with a fresh candidate: the rings, kept current
        # by the commit, give the paged call's bits
        q = dev_u16(S.normal_bf16(S.rng(6300 + seed, S.STREAM_Q), (L, B, Hkv, D)))
        kc = dev_u16(S.normal_bf16(S.rng(6400 + seed, S.STREAM_KCUR), (L, B, Hkv, D)))
        vc = dev_u16(S.normal_bf16(S.rng(6400 + seed, S.STREAM_VCUR), (L, B, Hkv, D)))
        lshape = P.Shape(L, B, Hkv, Hkv, D, mb, int(seq.max()) + 1, nb, layer_stride_kv=stride)
        wsl = torch.zeros(max(256, P.attn_workspace_size(lshape, n_sink, window)), dtype=torch.uint8, device="cuda")
        outs = []
        for use_ring in (False, True):
            out = torch.full((L, B, Hkv, D), float("nan"), device="cuda")
            lse = torch.full((L, B, Hkv), float("nan"), device="cuda")
            if use_ring:
                P.local_decode_attn_ring(lshape, P.inputs(q, None, None, None, dseq, D ** -0.5, kc, vc), kr, vr,
                                         n_sink, window, out, lse, wsl)
            else:
                P.local_decode_attn(lshape, P.inputs(q, dk, dv, dtable, dseq, D ** -0.5, kc, vc), n_sink, window,
                                    out, lse, wsl)
            torch.cuda.synchronize()
            outs.append((out, lse))
        assert torch.equal(outs[0][0].view(torch.int32), outs[1][0].view(torch.int32))
        assert torch.equal(outs[0][1].view(torch.int32), outs[1][1].view(torch.int32))
