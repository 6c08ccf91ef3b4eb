"""Pins of the decoder oracle (oracle/decoder.py) against closed forms,
library routines and invariants; CPU only."""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from oracle import attention as A
from oracle import decoder as OD
from oracle import gate as OG


def _bits(x):
    return S.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def test_rope_worked_example():
    """R1 of tests/golden/decoder_worked.txt."""
    x = np.array([1.0, 2.0, 3.0, 4.0])
    got = OD.rope(x, 2, 100.0)
    want = [1 * math.cos(2) - 3 * math.sin(2), 2 * math.cos(0.2) - 4 * math.sin(0.2),
            3 * math.cos(2) + 1 * math.sin(2), 4 * math.cos(0.2) + 2 * math.sin(0.2)]
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)
    np.testing.assert_array_equal(OD.rope(x, 0, 100.0), x)


def test_rope_is_a_relative_rotation():
    g = np.random.default_rng(3)
    q, k = g.standard_normal((2, 128))
    for m, n, sh in ((5, 2, 7), (100000, 3, 123456), (0, 0, 516000)):
        a = OD.rope(q, m, 1e6) @ OD.rope(k, n, 1e6)
        b = OD.rope(q, m + sh, 1e6) @ OD.rope(k, n + sh, 1e6)
        assert abs(a - b) < 1e-9 * (1 + abs(a))
        assert abs(np.linalg.norm(OD.rope(q, m, 1e6)) - np.linalg.norm(q)) < 1e-12


def test_round_bf16_ties_to_even_and_matches_torch():
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.0, 0.0, 1e-40, 65504.0, 1e38])
    got = OD.round_bf16(x)
    assert got[0] == 1.0 and got[1] == 1 + 2 ** -6 and got[2] == -1.0 and got[3] == 3.0
    y = np.random.default_rng(1).standard_normal(4096) * 10.0 ** np.random.default_rng(2).integers(-20, 20, 4096)
    ref = torch.from_numpy(y.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(OD.round_bf16(y), ref)


def test_dense_and_swiglu_match_torch():
    g = np.random.default_rng(4)
    W = _bits(g.standard_normal((10, 24)))
    x = g.standard_normal((3, 24))
    gain = 1 + 0.1 * g.standard_normal(24)
    r = g.standard_normal((3, 10))
    Wt = torch.from_numpy(A.bf16_to_f64(W))
    xt = torch.from_numpy(x)
    xn = torch.nn.functional.rms_norm(xt, (24,), torch.from_numpy(gain), eps=1e-5)
    np.testing.assert_allclose(OD.dense(W, x, gain, 1e-5, r), (torch.nn.functional.linear(xn, Wt) + torch.from_numpy(r)).numpy(),
                               rtol=1e-12, atol=1e-12)
    y = torch.nn.functional.linear(xn, Wt)
    want = torch.nn.functional.silu(y[:, :5]) * y[:, 5:]
    np.testing.assert_allclose(OD.swiglu(W, x, gain, 1e-5), want.numpy(), rtol=1e-12, atol=1e-12)
    # no gain: no normalisation, for both modes (the dense ABI's NULL norm gain)
    y0 = torch.nn.functional.linear(xt, Wt)
    np.testing.assert_allclose(OD.dense(W, x), y0.numpy(), rtol=1e-12, atol=1e-12)
    want0 = torch.nn.functional.silu(y0[:, :5]) * y0[:, 5:]
    np.testing.assert_allclose(OD.swiglu(W, x, None, 1e-5), want0.numpy(), rtol=1e-12, atol=1e-12)


def _worked_model():
    w = {"embed": _bits([[1, 1], [-1, 0.5], [0.5, 2]]),
         "attn_norm": np.ones((1, 2), np.float32),
         "w_qkv": _bits([[[1, 0], [0, 1], [1, 0], [0, 1], [2, 0], [0, -1]]]),
         "q_norm": np.ones((1, 2), np.float32), "k_norm": np.ones((1, 2), np.float32),
         "w_o": _bits([[[1, 0], [0, 1]]]),
         "mlp_norm": np.ones((1, 2), np.float32),
         "w_gu": _bits([[[1, 0], [0.5, 0]]]),
         "w_down": _bits([[[1], [0]]]),
         "final_norm": np.ones(2, np.float32)}
    return OD.Model(w, 1, 1, 2, eps=0.0, theta=1e6)


def test_decoder_layer_worked_example():
    """R2 of tests/golden/decoder_worked.txt."""
    m = _worked_model()
    # one-block caches in the ABI layouts (D = 2: one group of 2 dims); n = 1 reads nothing from them
    k = np.zeros((1, 1, 1, 1, 16, 2), np.uint16)
    v = np.zeros((1, 1, 1, 2, 16), np.uint16)
    table = np.zeros((1, 1), np.int32)
    h, kc, vc = m.forward([0], k, v, table, np.array([1]), A.full_set)
    s1 = 1 / (1 + math.exp(-math.sqrt(2)))
    mval = math.sqrt(2) * s1 * math.sqrt(2) / 2
    np.testing.assert_allclose(h[0], [3 + mval, 0.0], rtol=0, atol=1e-12)
    np.testing.assert_array_equal(A.bf16_to_f64(vc[0, 0, 0]), [2.0, -1.0])
    np.testing.assert_array_equal(A.bf16_to_f64(kc[0, 0, 0]), [1.0, 1.0])
    np.testing.assert_allclose(m.logits(h)[0], [math.sqrt(2), -math.sqrt(2), math.sqrt(2) / 2], atol=1e-12)
    assert OD.argmax(m.logits(h))[0] == 0


def _small(seed=1, L=2, d=128, Hq=4, Hkv=2, D=64, F=192, V=300, seq=(5, 40, 100)):
    w = S.decoder_weights(seed, L, d, Hq, Hkv, D, F, V)
    seq = np.array(seq, dtype=np.int32)
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq, None)
    k, v = S.kv_cache(seed, L, nb, Hkv, D)
    return OD.Model(w, Hq, Hkv, D), k, v, table, seq


def test_zero_layers_are_identities():
    m, k, v, table, seq = _small()
    for name in ("w_qkv", "w_o", "w_gu", "w_down"):
        m.w[name] = np.zeros_like(m.w[name])
    toks = np.array([3, 7, 11])
    h, kc, vc = m.forward(toks, k, v, table, seq, A.full_set)
    np.testing.assert_array_equal(h, m.embed(toks))
    assert not A.bf16_to_f64(kc).any() and not A.bf16_to_f64(vc).any()    # (+-0)


def test_local_equals_full_when_the_window_covers_the_history():
    m, k, v, table, seq = _small()
    toks = np.array([1, 2, 3])
    hf = m.forward(toks, k, v, table, seq, A.full_set)
    hl = m.forward(toks, k, v, table, seq, lambda n: A.local_set(n, 4, 200))
    for a, b in zip(hf, hl):
        np.testing.assert_array_equal(a, b)
    hs = m.forward(toks, k, v, table, seq, lambda n: A.local_set(n, 4, 24))
    assert not np.allclose(hs[0][2], hf[0][2])      # request 2 (n = 100) sees less


def test_subset_forward_matches_rows():
    m, k, v, table, seq = _small()
    toks = np.array([1, 2, 3])
    h, kc, vc = m.forward(toks, k, v, table, seq, A.full_set)
    hs, ks, vs = m.forward(toks, k, v, table, seq, A.full_set, requests=[2, 0])
    np.testing.assert_array_equal(hs[[0, 2]], h[[0, 2]])
    assert np.isnan(hs[1]).all()
    np.testing.assert_array_equal(ks[:, [0, 2]], kc[:, [0, 2]])


@pytest.mark.parametrize("flags", [(0, 0, 0), (1, 1, 1), (1, 0, 1)])
def test_oda_step_selects_the_branch(flags):
    m, k, v, table, seq = _small()
    toks = np.array([5, 6, 7])
    params = S.gate_params(2, "mlp", 128, 16)
    score = lambda hp, e, hl: OG.mlp_score(params, 128, 16, hl)
    hp = np.zeros((3, 128))
    r = OD.oda_step(m, toks, k, v, table, seq, 4, 24, score, hp, 0.0, forced=np.array(flags))
    hl = m.forward(toks, k, v, table, seq, lambda n: A.local_set(n, 4, 24))[0]
    hf = m.forward(toks, k, v, table, seq, A.full_set)[0]
    for b, f in enumerate(flags):
        np.testing.assert_array_equal(r["h"][b], hf[b] if f else hl[b])
    np.testing.assert_array_equal(r["flags"], flags)
    np.testing.assert_array_equal(r["logits"], m.logits(r["h"]))


def test_final_state_hand_worked():
    """RMSNorm with the final gain on a hand-worked row: h = (3, 4), gain
    (2, 0.5), eps = 0 -> mean(h^2) = 12.5, so the state is (6, 2) / sqrt(12.5)."""
    w = {"w_qkv": np.zeros((1, 1, 2), np.uint16), "embed": np.zeros((4, 2), np.uint16),
         "final_norm": np.array([2.0, 0.5], np.float32)}
    m = OD.Model(w, 1, 1, 2, eps=0.0)
    np.testing.assert_allclose(m.final_state(np.array([[3.0, 4.0]])), [[1.6970562748477140, 0.5656854249492380]],
                               rtol=1e-15)


def test_oda_step_feeds_the_head_final_normalised_states():
    """§2.1: the head's Local input is the final normalised Local hidden state;
    App. A.5: the state the step hands on (the next h_{t-1}) is the final
    normalised selected state, the one the vocabulary projection reads.  The
    score function sees exactly (h_prev as given, E(x_t), RMSNorm(h^L))."""
    m, k, v, table, seq = _small()
    toks = np.array([5, 6, 7])
    seen = {}

    def score(hp, e, hl):
        seen.update(hp=hp.copy(), e=e.copy(), hl=hl.copy())
        return np.array([1.0, -1.0, 1.0])

    hp = np.arange(3 * 128, dtype=np.float64).reshape(3, 128) / 100.0
    r = OD.oda_step(m, toks, k, v, table, seq, 4, 24, score, hp, 0.0)
    hl = m.forward(toks, k, v, table, seq, lambda n: A.local_set(n, 4, 24))[0]
    g = m.w["final_norm"].astype(np.float64)
    want = hl / np.sqrt(np.mean(hl * hl, axis=-1, keepdims=True) + m.eps) * g
    np.testing.assert_allclose(seen["hl"], want, rtol=1e-13, atol=0)
    np.testing.assert_array_equal(seen["hp"], hp)
    np.testing.assert_array_equal(seen["e"], m.embed(toks))
    hs = r["h"] / np.sqrt(np.mean(r["h"] ** 2, axis=-1, keepdims=True) + m.eps) * g
    np.testing.assert_allclose(r["h_state"], hs, rtol=1e-13, atol=0)
    np.testing.assert_array_equal(r["flags"], [1, 0, 1])
    # the gain matters: with a non-unit gain the raw and normalised inputs differ
    assert not np.allclose(seen["hl"], hl)


def test_argmax_first_index_and_nan():
    x = np.array([[1.0, 3.0, 3.0, np.nan], [np.nan] * 4, [-np.inf] * 4, [2.0, np.nan, 5.0, 5.0]])
    np.testing.assert_array_equal(OD.argmax(x), [1, -1, 0, 2])
