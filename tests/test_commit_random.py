"""Seeded random selected-state commits (App. A.5 commit equation) against
the oracle's commit: layer count, batch, KV heads, head width, lengths
(block boundaries included), per-request flags, with and without the Full
candidates, the length advance on or off, dense or padded layer strides."""
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
    mb = int(np.ceil(seq.max() / 16))
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
    shape = P.Shape(L, B, Hkv, Hkv, D, mb, int(seq.max()), nb, layer_stride_kv=stride)
    ws = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    P.commit_kv(shape, dk, dv, dev_i32(table), dseq, dev_u16(kl), dev_u16(vl),
                dev_u16(kf) if with_full else None, dev_u16(vf) if with_full else None,
                dev_i32(flags) if with_full else None, advance, ws)
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
