"""Pins of the oracle's whole decode step (oracle.step.decode_step) on the
CPU: Alg. 1's selection against attention written out independently here
(explicit position loops over the paged cache, torch softmax in fp64).

* threshold -inf: every request is flagged and the selected output is Full;
* threshold +inf: nothing is flagged, the output is Local and the Full part
  reads nothing (NaN rows);
* prescribed flags pick per request, and a nonfinite score sends a request
  to Full whatever the schedule says (§2.1, Alg. 1, App. B.7);
* a natively windowed Full uses the native window, not the whole history.
"""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from oracle import gate as OG
from oracle import step as OS

L, B, HQ, HKV, D = 2, 4, 4, 2, 16
SEQ = np.array([5, 40, 100, 33], dtype=np.int32)
SINK, WIN = 4, 24
DM, DT = 32, 8


def _problem(seed=3):
    q = S.normal_bf16(S.rng(seed, S.STREAM_Q), (L, B, HQ, D))
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), SEQ, None, permute=True)
    k, v = S.kv_cache(seed, L, nb, HKV, D)
    params = S.gate_params(seed, "paper", DM, DT)
    h, e, hl = (x[0].astype(np.float64) for x in S.gate_inputs(seed, 1, B, DM))
    return q, k, v, table, params, h, e, hl


def _bf(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _attention(q, k, v, table, member):
    """out[l][b][h][:] over the positions j < n with member(n, j), written
    out position by position from the paged layouts."""
    G = HQ // HKV
    out = np.zeros((L, B, HQ, D))
    for l in range(L):
        for b in range(B):
            n = int(SEQ[b])
            pos = [j for j in range(n) if member(n, j)]
            for h in range(HQ):
                g = h // G
                K = np.array([_bf(k[l, table[b, j // 16], g, :, j % 16, :]).reshape(D) for j in pos])
                V = np.array([_bf(v[l, table[b, j // 16], g, :, j % 16]) for j in pos])
                z = torch.from_numpy(K @ _bf(q[l, b, h]) / math.sqrt(D))
                w = torch.softmax(z, dim=0).numpy()
                out[l, b, h] = w @ V
    return out


def _local(n, j):
    return j < SINK or j >= n - WIN


def _full(n, j):
    return True


def _step(tau, forced=None, native_window=0, hl=None):
    q, k, v, table, params, h, e, hl0 = _problem()
    return OS.decode_step(q, k, v, table, SEQ, 1.0 / math.sqrt(D), SINK, WIN, "paper", params, DM, DT, 1e-6,
                          h, e, hl0 if hl is None else hl, tau, forced=forced, native_window=native_window)


def test_threshold_minus_inf_selects_full_for_every_request():
    q, k, v, table, *_ = _problem()
    r = _step(-math.inf)
    assert r["flags"].tolist() == [1] * B and r["n_work"] == B and list(r["work_list"]) == list(range(B))
    np.testing.assert_allclose(r["out"], _attention(q, k, v, table, _full), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["out_local"], _attention(q, k, v, table, _local), rtol=0, atol=1e-12)


def test_threshold_plus_inf_selects_local_and_reads_no_history():
    q, k, v, table, *_ = _problem()
    r = _step(math.inf)
    assert r["flags"].tolist() == [0] * B and r["n_work"] == 0 and len(r["work_list"]) == 0
    np.testing.assert_allclose(r["out"], _attention(q, k, v, table, _local), rtol=0, atol=1e-12)
    assert np.isnan(r["out_full"]).all()


def test_mixed_prescribed_flags_select_per_request():
    q, k, v, table, *_ = _problem()
    forced = np.array([1, 0, 0, 1], dtype=np.int32)
    r = _step(0.0, forced=forced)
    full = _attention(q, k, v, table, _full)
    loc = _attention(q, k, v, table, _local)
    assert r["flags"].tolist() == [1, 0, 0, 1] and list(r["work_list"]) == [0, 3]
    for b in range(B):
        np.testing.assert_allclose(r["out"][:, b], (full if forced[b] else loc)[:, b], rtol=0, atol=1e-12)
    # the lse rows follow the same selection
    for b in range(B):
        want = r["lse_full"][:, b] if forced[b] else r["lse_local"][:, b]
        np.testing.assert_array_equal(r["lse"][:, b], want)


def test_threshold_splits_requests_by_score():
    q, k, v, table, params, h, e, hl = _problem()
    score = OG.paper_head_score(params, DM, DT, 1e-6, h, e, hl)
    tau = float(np.sort(score)[1] + np.sort(score)[2]) / 2          # two above, two below
    r = _step(tau)
    np.testing.assert_array_equal(r["score"], score)
    want = (score > tau).astype(np.int32)
    assert r["flags"].tolist() == want.tolist() and want.sum() == 2
    full = _attention(q, k, v, table, _full)
    loc = _attention(q, k, v, table, _local)
    for b in range(B):
        np.testing.assert_allclose(r["out"][:, b], (full if want[b] else loc)[:, b], rtol=0, atol=1e-12)


def test_nonfinite_score_goes_to_full_even_under_a_schedule():
    q, k, v, table, params, h, e, hl = _problem()
    hl = hl.copy()
    hl[2, 5] = np.nan
    r = _step(0.0, forced=np.array([0, 0, 0, 0], dtype=np.int32), hl=hl)
    assert r["flags"].tolist() == [0, 0, 1, 0]
    np.testing.assert_allclose(r["out"][:, 2], _attention(q, k, v, table, _full)[:, 2], rtol=0, atol=1e-12)


@pytest.mark.parametrize("native", [16, 30])
def test_native_window_full(native):
    q, k, v, table, *_ = _problem()
    r = _step(-math.inf, native_window=native)
    want = _attention(q, k, v, table, lambda n, j: j >= n - native)
    np.testing.assert_allclose(r["out"], want, rtol=0, atol=1e-12)
