"""Seeded random problems for the decoder kernels around the hot path against
the fp64 oracle: dense layers (widths with ragged chunk tails, batches over
several tiles, RMSNorm, residual, SwiGLU, selection lists), q/k RMSNorm +
rotary (head widths, GQA groups, positions, lists) and the greedy argmax
(lengths, ties, NaN rows), with the tolerances of test_decoder_parity.py."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import dev_f32, dev_i32, dev_u16, need_gpu
from oracle import decoder as OD
from test_decoder_parity import DENSE_REL, _bf16_close

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(40))
def test_random_dense(seed):
    P = need_gpu()
    g = np.random.default_rng(7000 + seed)
    K = 8 * int(g.integers(1, 640))
    N = int(g.integers(1, 300))
    B = int(g.choice([1, 2, 3, 7, 8, 9, 16, 33, 70]))
    swiglu = bool(g.random() < 0.35)
    norm = bool(g.random() < 0.6)
    res = (not swiglu) and bool(g.random() < 0.5)
    listed = bool(g.random() < 0.3)
    rows = 2 * N if swiglu else N
    gen = S.rng(7000 + seed, S.STREAM_DECODER)
    W = S.normal_bf16(gen, (rows, K), K ** -0.5)
    x = gen.standard_normal((B, K)).astype(np.float32)
    gain = (1 + 0.02 * gen.standard_normal(K)).astype(np.float32) if norm else None
    r = gen.standard_normal((B, N)).astype(np.float32) if res else None
    sel = sorted(g.choice(B, size=int(g.integers(0, B + 1)), replace=False).tolist(), reverse=True) \
        if listed else list(range(B))
    desc = P.dense_desc(K, N, P.DENSE_SWIGLU if swiglu else P.DENSE_PLAIN, dev_u16(W),
                        dev_f32(gain) if norm else None, 1e-6)
    y = torch.full((B, N), 7.0, device="cuda")
    wl = dev_i32(sel + [0] * (B - len(sel))) if listed else None
    nw = dev_i32([len(sel)]) if listed else None
    P.dense_bf16(desc, B, dev_f32(x), dev_f32(r) if res else None, y, wl, nw)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    if sel:
        ref = OD.swiglu(W, x[sel], gain, 1e-6) if swiglu else OD.dense(W, x[sel], gain, 1e-6,
                                                                       r[sel] if res else None)
        scale = max(1.0, float(np.abs(ref).max()))
        err = float(np.abs(got[sel] - ref).max())
        assert err <= DENSE_REL * scale, (K, N, B, swiglu, norm, res, listed, err)
    others = [b for b in range(B) if b not in sel]
    assert np.all(got[others] == 7.0)


@pytest.mark.parametrize("seed", range(20))
def test_random_qk_norm_rope(seed):
    P = need_gpu()
    g = np.random.default_rng(8000 + seed)
    D = 2 * int(g.integers(1, 65))
    Hkv = int(g.integers(1, 9))
    Hq = Hkv * int(g.choice([1, 2, 4]))
    B = int(g.integers(1, 10))
    gains = bool(g.random() < 0.7)
    listed = bool(g.random() < 0.3)
    gen = S.rng(8000 + seed, S.STREAM_DECODER)
    qkv = (3 * gen.standard_normal((B, (Hq + 2 * Hkv) * D))).astype(np.float32)
    qg = (1 + 0.02 * gen.standard_normal(D)).astype(np.float32) if gains else None
    kg = (1 + 0.02 * gen.standard_normal(D)).astype(np.float32) if gains else None
    seq = g.integers(1, 600000, size=B).astype(np.int32)
    sel = sorted(g.choice(B, size=int(g.integers(0, B + 1)), replace=False).tolist()) if listed else list(range(B))
    q = torch.full((B, Hq, D), 5.0, dtype=torch.bfloat16, device="cuda")
    k = torch.full((B, Hkv, D), 5.0, dtype=torch.bfloat16, device="cuda")
    v = torch.full((B, Hkv, D), 5.0, dtype=torch.bfloat16, device="cuda")
    wl = dev_i32(sel + [0] * (B - len(sel))) if listed else None
    nw = dev_i32([len(sel)]) if listed else None
    P.qk_norm_rope(B, Hq, Hkv, D, dev_f32(qkv), dev_f32(qg) if gains else None, dev_f32(kg) if gains else None,
                   1e-6, 1e6, dev_i32(seq), q, k, v, wl, nw)
    torch.cuda.synchronize()
    bits = lambda t: t.cpu().view(torch.int16).numpy().view(np.uint16)
    if sel:
        rq, rk, rv = OD.qk_norm_rope(qkv[sel], Hq, Hkv, D, qg, kg, 1e-6, 1e6, seq[sel] - 1)
        _bf16_close(bits(q)[sel], OD.bf16_bits(rq), f"q (D={D})")
        _bf16_close(bits(k)[sel], OD.bf16_bits(rk), f"k (D={D})")
        np.testing.assert_array_equal(bits(v)[sel], OD.bf16_bits(rv))
    others = [b for b in range(B) if b not in sel]
    assert torch.all(q.cpu()[others] == 5.0)


@pytest.mark.parametrize("seed", range(20))
def test_random_argmax(seed):
    P = need_gpu()
    g = np.random.default_rng(9000 + seed)
    B = int(g.integers(1, 9))
    n = 4 * int(g.integers(1, 50000))
    x = g.standard_normal((B, n)).astype(np.float32)
    for b in range(B):
        kind = g.integers(0, 4)
        if kind == 1:                       # a tie between two maxima
            i, j = sorted(g.choice(n, size=2, replace=n < 2) if n > 1 else [0, 0])
            x[b, i] = x[b, j] = 40.0
        elif kind == 2:                     # NaN entries
            x[b, g.choice(n, size=max(1, n // 7), replace=False)] = np.nan
        elif kind == 3:                     # constant row
            x[b] = 1.5
    idx = torch.zeros(B, dtype=torch.int32, device="cuda")
    P.argmax(B, n, dev_f32(x), idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(idx.cpu().numpy(), OD.argmax(x))
