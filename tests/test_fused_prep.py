"""The attention calls with the current token prepared in the call
(oda_local_decode_attn_qkv, oda_full_decode_attn_qkv).

Against oda_qk_norm_rope followed by the plain call on the same inputs, the
results must be bit-identical (out, lse, and the candidate K/V written for the
commit): both run the same per-head preparation code and then the same
attention arithmetic.  Cases cover D = 64 / 128, GQA groups 1 to 16, forced
multi-split plans (the merge reads the prepared candidate), Local and Full with
every request, with flags and with a work list (empty, and a subset), and
positions up to 516,787.  One small case is also checked against the fp64
oracle directly: its q/k/v preparation rounded to bf16, then attention with the
candidate as position n - 1."""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from harness import check_close, dev_f32, dev_i32, dev_u16, need_gpu
from oracle import attention as OA
from oracle import decoder as OD

pytestmark = pytest.mark.gpu

EPS, THETA = 1e-6, 1e6
SENTINEL = 7.0


def _problem(P, seed, D, Hq, Hkv, seq, gains):
    B = len(seq)
    seq = np.asarray(seq, dtype=np.int32)
    mb = int(math.ceil(seq.max() / 16))
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq, mb, permute=True)
    ks, vs = S.kv_cache_shapes(1, nb, Hkv, D)
    k = torch.empty(ks, dtype=torch.bfloat16, device="cuda")
    v = torch.empty(vs, dtype=torch.bfloat16, device="cuda")
    S.fill_normal_bf16_(k, seed, S.STREAM_K)
    S.fill_normal_bf16_(v, seed, S.STREAM_V)
    g = S.rng(seed, S.STREAM_DECODER)
    qkv = (3 * g.standard_normal((B, (Hq + 2 * Hkv) * D))).astype(np.float32)
    qg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32) if gains else None
    kg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32) if gains else None
    shape = P.Shape(1, B, Hq, Hkv, D, mb, int(seq.max()), nb, 0)
    return dict(B=B, seq=seq, table=table, nb=nb, mb=mb, k=k, v=v, qkv=qkv, qg=qg, kg=kg, shape=shape,
                dtable=dev_i32(table), dseq=dev_i32(seq))


def _run_both(P, pr, D, Hq, Hkv, branch, s=4, W=64, split_blocks=0, select="all", listed=None, native=0):
    """(unfused, fused) results: out, lse, k candidate, v candidate (device tensors)."""
    B = pr["B"]
    shape = P.Shape(1, B, Hq, Hkv, D, pr["mb"], int(pr["seq"].max()), pr["nb"], split_blocks)
    qkv = dev_f32(pr["qkv"])
    qg = dev_f32(pr["qg"]) if pr["qg"] is not None else None
    kg = dev_f32(pr["kg"]) if pr["kg"] is not None else None
    flags = wl = nw = None
    if select == "flags":
        f = np.zeros(B, np.int32)
        f[listed] = 1
        flags = dev_i32(f)
    elif select == "list":
        wl = dev_i32(list(listed) + [0] * (B - len(listed)))
        nw = dev_i32([len(listed)])
    scale = 1.0 / math.sqrt(D)
    res = []
    for fused in (False, True):
        out = torch.full((1, B, Hq, D), SENTINEL, device="cuda")
        lse = torch.full((1, B, Hq), SENTINEL, device="cuda")
        kc = torch.full((1, B, Hkv, D), SENTINEL, dtype=torch.bfloat16, device="cuda")
        vc = torch.full((1, B, Hkv, D), SENTINEL, dtype=torch.bfloat16, device="cuda")
        sw, ww = (s, W) if branch == "local" else (0, native)
        ws = torch.zeros(max(256, P.attn_workspace_size(shape, sw, ww)), dtype=torch.uint8, device="cuda")
        if fused:
            prep = P.qkv_prep(qkv, qg, kg, EPS, THETA, kc, vc)
            inp = P.inputs(None, pr["k"], pr["v"], pr["dtable"], pr["dseq"], scale)
            if branch == "local":
                P.prepare_local_qkv(shape, inp, prep, s, W, out, lse, ws)()
            else:
                P.prepare_full_qkv(shape, inp, prep, native, flags, wl, nw, out, lse, ws)()
        else:
            q = torch.full((1, B, Hq, D), SENTINEL, dtype=torch.bfloat16, device="cuda")
            # the unfused decoder prepares exactly the requests it attends
            P.qk_norm_rope(B, Hq, Hkv, D, qkv, qg, kg, EPS, THETA, pr["dseq"], q[0], kc[0], vc[0], wl, nw)
            if select == "flags":   # qk_norm_rope takes no flags: keep only the flagged rows' candidates
                keep = torch.zeros(B, dtype=torch.bool, device="cuda")
                keep[list(listed)] = True
                kc[0][~keep] = SENTINEL
                vc[0][~keep] = SENTINEL
            inp = P.inputs(q, pr["k"], pr["v"], pr["dtable"], pr["dseq"], scale, kc, vc)
            if branch == "local":
                P.local_decode_attn(shape, inp, s, W, out, lse, ws)
            else:
                P.full_decode_attn(shape, inp, native, flags, wl, nw, out, lse, ws)
        torch.cuda.synchronize()
        res.append((out.cpu(), lse.cpu(), kc.cpu(), vc.cpu()))
    return res


def _assert_identical(res):
    """Bit patterns equal (NaN rows of invalid requests included)."""
    (ou, lu, ku, vu), (of, lf, kf, vf) = res
    assert torch.equal(ou.view(torch.int32), of.view(torch.int32)), float((ou - of).abs().nan_to_num().max())
    assert torch.equal(lu.view(torch.int32), lf.view(torch.int32))
    assert torch.equal(ku.view(torch.int16), kf.view(torch.int16))
    assert torch.equal(vu.view(torch.int16), vf.view(torch.int16))


@pytest.mark.parametrize("D,Hq,Hkv,seq,gains,split", [
    (128, 16, 8, [5, 300, 2100], True, 0),        # the decoder's heads (G = 2)
    (64, 8, 2, [1, 70, 131072], False, 6),        # G = 4, forced 6-block splits (in-launch merge)
    (128, 16, 1, [516788], True, 0),              # G = 16, the longest position
    (128, 8, 8, [33, 17], True, 2),               # G = 1, 2-block splits
])
def test_local_fused_equals_qk_norm_rope_then_local(D, Hq, Hkv, seq, gains, split):
    P = need_gpu()
    pr = _problem(P, 11 + D + Hq, D, Hq, Hkv, seq, gains)
    res = _run_both(P, pr, D, Hq, Hkv, "local", s=4, W=2048 if max(seq) > 4096 else 64, split_blocks=split)
    _assert_identical(res)
    assert not torch.isnan(res[1][0]).any()


@pytest.mark.parametrize("select,listed,split", [("all", None, 0), ("flags", [1, 2], 0), ("list", [2, 0], 6),
                                                 ("list", [], 0), ("all", None, 4)])
def test_full_fused_equals_qk_norm_rope_then_full(select, listed, split):
    P = need_gpu()
    D, Hq, Hkv = 128, 16, 8
    pr = _problem(P, 5, D, Hq, Hkv, [40, 2000, 9000], True)
    res = _run_both(P, pr, D, Hq, Hkv, "full", split_blocks=split, select=select, listed=listed)
    _assert_identical(res)
    out_f = res[1][0]
    attended = range(3) if select == "all" else listed
    for b in range(3):   # only the selected rows (and candidates) are written
        if b in attended:
            assert not torch.isnan(out_f[0, b]).any() and not (out_f[0, b] == SENTINEL).all()
        else:
            assert (out_f[0, b] == SENTINEL).all()
            assert (res[1][2][0, b].float() == SENTINEL).all()


def test_native_window_full_fused():
    P = need_gpu()
    D, Hq, Hkv = 64, 4, 2
    pr = _problem(P, 9, D, Hq, Hkv, [10, 500], False)
    _assert_identical(_run_both(P, pr, D, Hq, Hkv, "full", native=48))


@pytest.mark.parametrize("branch", ["local", "full"])
def test_invalid_length_gives_nan_rows_both_ways(branch):
    """A length above max_seq_len addresses no history in either path: that
    request's rows are NaN, its candidate is still prepared (as
    oda_qk_norm_rope prepares it), and the other requests are unaffected."""
    P = need_gpu()
    D, Hq, Hkv = 64, 8, 2
    pr = _problem(P, 13, D, Hq, Hkv, [40, 300, 77], True)
    pr["dseq"][1] = 301                      # above the shape's max_seq_len (300)
    res = _run_both(P, pr, D, Hq, Hkv, branch, split_blocks=2)
    _assert_identical(res)
    out = res[1][0]
    assert torch.isnan(out[0, 1]).all()
    assert not torch.isnan(out[0, 0]).any() and not torch.isnan(out[0, 2]).any()


def test_fused_local_matches_the_oracle():
    """q/k/v prepared by the oracle in fp64 and rounded to bf16, then attention
    over S^L with the candidate at position n - 1.  The two sides round the
    prepared values themselves, so a rare element may sit one bf16 step apart;
    the attention bar absorbs that."""
    P = need_gpu()
    D, Hq, Hkv, s, W = 64, 4, 2, 4, 16
    seq = np.array([3, 40, 97], dtype=np.int32)
    B = len(seq)
    mb = int(math.ceil(seq.max() / 16))
    table, nb = S.paged_block_table(S.rng(21, S.STREAM_TABLE), seq, mb, permute=True)
    k, v = S.kv_cache(21, 1, nb, Hkv, D)
    g = S.rng(21, S.STREAM_DECODER)
    qkv = (3 * g.standard_normal((B, (Hq + 2 * Hkv) * D))).astype(np.float32)
    qg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32)
    kg = (1 + 0.02 * g.standard_normal(D)).astype(np.float32)
    shape = P.Shape(1, B, Hq, Hkv, D, mb, int(seq.max()), nb, 0)
    out = torch.zeros((1, B, Hq, D), device="cuda")
    lse = torch.zeros((1, B, Hq), device="cuda")
    kc = torch.zeros((1, B, Hkv, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    ws = torch.zeros(max(256, P.attn_workspace_size(shape, s, W)), dtype=torch.uint8, device="cuda")
    inp = P.inputs(None, dev_u16(k), dev_u16(v), dev_i32(table), dev_i32(seq), 1 / math.sqrt(D))
    P.prepare_local_qkv(shape, inp, P.qkv_prep(dev_f32(qkv), dev_f32(qg), dev_f32(kg), EPS, THETA, kc, vc),
                        s, W, out, lse, ws)()
    torch.cuda.synchronize()
    rq, rk, rv = OD.qk_norm_rope(qkv, Hq, Hkv, D, qg, kg, EPS, THETA, seq - 1)
    q_bits = OD.bf16_bits(rq).reshape(1, B, Hq, D)
    k_bits = OD.bf16_bits(rk).reshape(1, B, Hkv, D)
    v_bits = OD.bf16_bits(rv).reshape(1, B, Hkv, D)
    ref, ref_lse, _ = OA.decode_attention(q_bits, k, v, table, seq, lambda n: OA.local_set(n, s, W), 1 / math.sqrt(D),
                                          k_cur=k_bits, v_cur=v_bits)
    # one-step rounding differences of q or k move a score by up to ~1e-3, so
    # the target's bar applies here, not the internal 1e-4 one
    check_close(out.cpu().numpy(), ref, internal=False)
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, rtol=0, atol=2e-3)
    got_v = vc.cpu().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got_v, v_bits)          # v: one rounding of the input
