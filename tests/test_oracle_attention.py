"""Pins of the fp64 attention oracle against what the paper and the
mathematics fix (no GPU)."""
import math
import os

import numpy as np
import pytest
import torch

import oda_synth as S
from oracle import attention as A

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _parse_ranges(txt):
    out = []
    for part in txt.split(","):
        part = part.strip()
        if "-" in part:
            a, b = part.split("-")
            out += list(range(int(a), int(b) + 1))
        elif part:
            out.append(int(part))
    return out


def _golden_sets():
    rows = []
    with open(os.path.join(GOLDEN, "access_sets.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split("|")
            t, s, w = (int(x) for x in lhs.split())
            rows.append((t, s, w, _parse_ranges(rhs)))
    return rows


@pytest.mark.parametrize("t,s,w,expected", _golden_sets())
def test_local_set_matches_hand_worked_equation(t, s, w, expected):
    # paper positions are 1-based; the oracle's are 0-based with n = t
    got = (A.local_set(t, s, w) + 1).tolist()
    assert got == expected


def test_local_equals_full_through_2052_and_differs_at_2053():
    # App. A.3: with s=4, w=2048 the sets coincide through position 2,052
    for t in (1, 2, 4, 5, 100, 2048, 2049, 2051, 2052):
        assert np.array_equal(A.local_set(t, 4, 2048), A.full_set(t))
    loc = A.local_set(2053, 4, 2048)
    assert len(loc) == 2052 and 4 not in loc          # position 5 (0-based 4) dropped
    for t in (2053, 5000, 131072):
        assert len(A.local_set(t, 4, 2048)) == 2052      # s + w, App. A.5


def _tiny_problem(seed, L=2, B=3, Hq=8, Hkv=2, D=64, seq=(1, 23, 70), permute=True, cur=False):
    g = S.rng(seed, S.STREAM_Q)
    q = S.normal_bf16(g, (L, B, Hq, D))
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq, permute=permute, extra_blocks=3)
    k, v = S.kv_cache(seed, L, nb, Hkv, D)
    kc = vc = None
    if cur:
        kc = S.normal_bf16(S.rng(seed, S.STREAM_KCUR), (L, B, Hkv, D))
        vc = S.normal_bf16(S.rng(seed, S.STREAM_VCUR), (L, B, Hkv, D))
    return q, k, v, table, np.array(seq, dtype=np.int32), kc, vc


def _logical_kv(k, v, table, l, b, g, n, kc=None, vc=None):
    """Contiguous [n][D] K/V of one request, read cell by cell from the layout."""
    D = k.shape[3] * 8
    K = np.zeros((n, D))
    V = np.zeros((n, D))
    for p in range(n):
        phys = table[b][p // 16]
        for d in range(D):
            K[p, d] = A.bf16_to_f64(k[l, phys, g, d // 8, p % 16, d % 8]).item()
            V[p, d] = A.bf16_to_f64(v[l, phys, g, d, p % 16]).item()
    if kc is not None:
        K[n - 1] = A.bf16_to_f64(kc[l, b, g])
        V[n - 1] = A.bf16_to_f64(vc[l, b, g])
    return K, V


@pytest.mark.parametrize("cur", [False, True])
@pytest.mark.parametrize("s,w", [(4, 16), (0, 5), (2, 1), (0, 1 << 30)])
def test_brute_force_vs_torch_sdpa(cur, s, w):
    """P9: masked softmax attention equals torch's SDPA in fp64 with a boolean
    mask and GQA expanded by repeat_interleave."""
    q, k, v, table, seq, kc, vc = _tiny_problem(7, cur=cur)
    L, B, Hq, D = q.shape
    Hkv = k.shape[2]
    scale = 1.0 / math.sqrt(D)
    out, lse, counts = A.decode_attention(q, k, v, table, seq, lambda n: A.local_set(n, s, w), scale,
                                          k_cur=kc, v_cur=vc)
    for l in range(L):
        for b in range(B):
            n = int(seq[b])
            Ks, Vs = [], []
            for g in range(Hkv):
                K, V = _logical_kv(k, v, table, l, b, g, n, kc, vc)
                Ks.append(K)
                Vs.append(V)
            Kt = torch.tensor(np.stack(Ks)).repeat_interleave(Hq // Hkv, 0)    # [Hq][n][D]
            Vt = torch.tensor(np.stack(Vs)).repeat_interleave(Hq // Hkv, 0)
            qt = torch.tensor(A.bf16_to_f64(q[l, b]))[:, None, :]             # [Hq][1][D]
            mask = torch.zeros(1, n, dtype=torch.bool)
            for p in range(n):
                mask[0, p] = (p < min(s, n)) or (p >= n - w)
            ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, attn_mask=mask, scale=scale)
            np.testing.assert_allclose(out[l, b], ref[:, 0].numpy(), rtol=1e-12, atol=1e-12)
            assert counts[b] == int(mask.sum())


def test_single_position_returns_v0_exactly():
    """P5: with t = 1 the only attended position is the current token."""
    q, k, v, table, seq, _, _ = _tiny_problem(3, seq=(1, 1, 1))
    out, lse, _ = A.decode_attention(q, k, v, table, seq, A.full_set, 0.125)
    for l in range(q.shape[0]):
        for b in range(q.shape[1]):
            for h in range(q.shape[2]):
                g = h // (q.shape[2] // k.shape[2])
                phys = table[b][0]
                assert np.array_equal(out[l, b, h], A.bf16_to_f64(v[l, phys, g, :, 0]))
                K0 = A.bf16_to_f64(k[l, phys, g, :, 0, :].reshape(-1))
                assert lse[l, b, h] == pytest.approx(0.125 * float(A.bf16_to_f64(q[l, b, h]) @ K0), abs=1e-12)


def test_constant_keys_give_mean_of_values():
    """P6: equal logits -> uniform weights: o = mean V over S, lse = z + ln|S|."""
    q, k, v, table, seq, _, _ = _tiny_problem(5, seq=(40, 77, 3))
    k[:] = S.f32_to_bf16_bits(np.float32(0.5))
    s, w = 4, 9
    out, lse, counts = A.decode_attention(q, k, v, table, seq, lambda n: A.local_set(n, s, w), 0.1)
    D = q.shape[3]
    for b in range(3):
        n = int(seq[b])
        pos = sorted(set(range(min(s, n))) | set(range(max(0, n - w), n)))
        for l in range(q.shape[0]):
            for h in range(q.shape[2]):
                g = h // 4
                Vm = np.mean([[A.bf16_to_f64(v[l, table[b][p // 16], g, d, p % 16]).item() for d in range(D)]
                              for p in pos], axis=0)
                np.testing.assert_allclose(out[l, b, h], Vm, rtol=1e-12, atol=1e-13)
                z = 0.1 * 0.5 * float(np.sum(A.bf16_to_f64(q[l, b, h])))
                assert lse[l, b, h] == pytest.approx(z + math.log(len(pos)), abs=1e-11)


def test_weights_sum_to_one_and_match_lse():
    """P4: sum_j exp(z_j - lse) = 1."""
    q, k, v, table, seq, _, _ = _tiny_problem(11)
    scale = 0.3
    out, lse, counts, W = A.decode_attention(q, k, v, table, seq, lambda n: A.local_set(n, 4, 20), scale,
                                             return_weights=True)
    for (l, b, h), (pos, w) in W.items():
        assert abs(np.sum(w) - 1.0) < 1e-12
        g = h // 4
        K = A.key_rows(k, table, l, b, g, pos)
        z = scale * (K @ A.bf16_to_f64(q[l, b, h]))
        assert abs(np.sum(np.exp(z - lse[l, b, h])) - 1.0) < 1e-12


@pytest.mark.parametrize("n", [1, 5, 20, 23, 24, 30])
def test_local_equals_full_when_window_covers_context(n):
    """P1: s + w >= n makes S^L = S^F, so both results are identical."""
    q, k, v, table, _, _, _ = _tiny_problem(13, seq=(30, 30, 30))
    seq = np.array([n, n, n], dtype=np.int32)
    full, lf, _ = A.decode_attention(q, k, v, table, seq, A.full_set, 0.125)
    for s, w in ((4, n - 4), (0, n), (n, 1), (4, 1 << 20)):
        if s + w < n:
            continue
        loc, ll, _ = A.decode_attention(q, k, v, table, seq, lambda m: A.local_set(m, s, w), 0.125)
        assert np.array_equal(loc, full) and np.array_equal(ll, lf)


def test_paged_equals_contiguous_layout():
    """P8: a permuted block table and the identity one give identical results."""
    qa, ka, va, ta, seq, _, _ = _tiny_problem(17, permute=False)
    qb, kb, vb, tb, _, _, _ = _tiny_problem(17, permute=True)
    # move the identity-table contents into the permuted blocks
    kb = np.zeros_like(ka)
    vb = np.zeros_like(va)
    for b in range(len(seq)):
        for i in range((int(seq[b]) + 15) // 16):
            kb[:, tb[b][i]] = ka[:, ta[b][i]]
            vb[:, tb[b][i]] = va[:, ta[b][i]]
    f = lambda n: A.local_set(n, 2, 33)
    oa = A.decode_attention(qa, ka, va, ta, seq, f, 0.2)
    ob = A.decode_attention(qa, kb, vb, tb, seq, f, 0.2)
    assert np.array_equal(oa[0], ob[0]) and np.array_equal(oa[1], ob[1])


def test_combining_partials_of_any_partition_equals_unsplit():
    """P7: the stable-softmax combination of partials over a partition of S
    equals the unsplit result (online-softmax identity)."""
    g = np.random.default_rng(0)
    for n in (1, 2, 17, 100):
        q = g.standard_normal(32)
        K = g.standard_normal((n, 32)) * 3
        V = g.standard_normal((n, 32))
        o, lse, _ = A.attend(q, K, V, 0.7)
        cuts = sorted(set(g.integers(1, n, size=min(n - 1, 4)).tolist())) if n > 1 else []
        edges = [0] + cuts + [n]
        parts = [A.partial_attend(q, K[a:b], V[a:b], 0.7) for a, b in zip(edges[:-1], edges[1:])]
        o2, lse2 = A.combine_partials(parts)
        np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-13)
        assert abs(lse2 - lse) < 1e-12


@pytest.mark.parametrize("n,s,w", [(70, 4, 16), (70, 0, 16), (33, 4, 29), (200, 7, 50)])
def test_dominant_key_probes_fix_set_membership(n, s, w):
    """P10: a key aligned with q at position p dominates the softmax iff p is
    in the access set, so o ~ V_p exactly at the set's boundaries."""
    D, Hkv, Hq = 64, 1, 1
    seq = [n]
    table, nb = S.paged_block_table(S.rng(3, S.STREAM_TABLE), seq, permute=True)
    k, v = S.kv_cache(3, 1, nb, Hkv, D)
    k = (S.bf16_bits_to_f32(k) * 0.05).astype(np.float32)
    k = S.f32_to_bf16_bits(k)
    qf = np.ones(D, dtype=np.float32)
    q = S.f32_to_bf16_bits(qf).reshape(1, 1, 1, D)
    S_true = set(range(min(s, n))) | set(range(max(0, n - w), n))
    probes = {s - 1, s, n - w - 1, n - w, n - 1, 0}
    for p in sorted(x for x in probes if 0 <= x < n):
        kp = k.copy()
        phys = table[0][p // 16]
        kp[0, phys, 0, :, p % 16, :] = S.f32_to_bf16_bits(np.full((D // 8, 8), 2.0, np.float32))
        out, _, _ = A.decode_attention(q, kp, v, table, np.array(seq), lambda m: A.local_set(m, s, w), 1.0)
        vp = A.bf16_to_f64(v[0, phys, 0, :, p % 16])
        hit = np.max(np.abs(out[0, 0, 0] - vp)) < 1e-6
        assert hit == (p in S_true), (p, hit)


def test_current_candidate_equals_cached_current_token():
    """k_cur/v_cur supply position n-1 (App. A.5); if they hold the same row as
    the cache, the result is unchanged."""
    q, k, v, table, seq, _, _ = _tiny_problem(19, seq=(1, 16, 17))
    L, B, Hq, D = q.shape
    Hkv = k.shape[2]
    kc = np.zeros((L, B, Hkv, D), np.uint16)
    vc = np.zeros((L, B, Hkv, D), np.uint16)
    for b in range(B):
        p = int(seq[b]) - 1
        phys = table[b][p // 16]
        kc[:, b] = k[:, phys, :, :, p % 16, :].reshape(L, Hkv, D)
        vc[:, b] = v[:, phys, :, :, p % 16]
    f = lambda n: A.local_set(n, 4, 8)
    a = A.decode_attention(q, k, v, table, seq, f, 0.2)
    # scribble over the cached current rows: they must not be read any more
    k2, v2 = k.copy(), v.copy()
    for b in range(B):
        p = int(seq[b]) - 1
        k2[:, table[b][p // 16], :, :, p % 16, :] = 0x7FC0
        v2[:, table[b][p // 16], :, :, p % 16] = 0x7FC0
    bres = A.decode_attention(q, k2, v2, table, seq, f, 0.2, k_cur=kc, v_cur=vc)
    np.testing.assert_allclose(bres[0], a[0], rtol=1e-12, atol=1e-14)


def test_commit_appends_selected_candidate():
    """App. A.5 commit equation: after committing, the cache holds the selected
    candidate at position n-1, so attending without the candidate gives what
    attending with it gave; the unselected branch's candidate is nowhere."""
    from oracle import step as OS
    q, k, v, table, seq, kc, vc = _tiny_problem(23, seq=(3, 16, 40), cur=True)
    kf = S.normal_bf16(S.rng(99, S.STREAM_KCUR), kc.shape)
    vf = S.normal_bf16(S.rng(99, S.STREAM_VCUR), vc.shape)
    flags = np.array([0, 1, 0])
    f = lambda n: A.local_set(n, 2, 9)
    before_l = A.decode_attention(q, k, v, table, seq, f, 0.3, k_cur=kc, v_cur=vc)
    before_f = A.decode_attention(q, k, v, table, seq, f, 0.3, k_cur=kf, v_cur=vf)
    k2, v2, s2 = k.copy(), v.copy(), seq.copy()
    OS.commit(k2, v2, table, s2, kc, vc, kf, vf, flags)
    assert s2.tolist() == [4, 17, 41]
    after = A.decode_attention(q, k2, v2, table, seq, f, 0.3)
    for b in range(3):
        want = before_f if flags[b] else before_l
        np.testing.assert_array_equal(after[0][:, b], want[0][:, b])
        p = int(seq[b]) - 1
        src = kf if flags[b] else kc
        assert np.array_equal(k2[:, table[b][p // 16], :, :, p % 16, :].reshape(src[:, b].shape), src[:, b])
    # nothing else changed
    mask = np.ones(k.shape[:2] + k.shape[2:], bool)
    for b in range(3):
        p = int(seq[b]) - 1
        mask[:, table[b][p // 16], :, :, p % 16, :] = False
    assert np.array_equal(k2[mask], k[mask])
