"""Pins of the fp64 recall-gate oracle (no GPU)."""
import math

import numpy as np
import pytest
import torch

import oda_synth as S
from oracle import gate as Gt


def test_parameter_count_matches_paper():
    """P11: App. A.2 states 28,325,889 parameters for d = 2048, tower 1024."""
    assert Gt.param_count(Gt.paper_head_shapes(2048, 1024)) == 28_325_889
    # the synthetic generator packs the same number of values
    assert sum(c for _, _, c in S.paper_head_segments(2048, 1024)) == 28_325_889


def test_synth_and_oracle_packing_orders_agree():
    a = [(n, int(np.prod(s))) for n, s in Gt.paper_head_shapes(64, 16)]
    b = [(n, c) for n, _, c in S.paper_head_segments(64, 16)]
    assert a == b
    a = [(n, int(np.prod(s))) for n, s in Gt.mlp_shapes(64, 16)]
    b = [(n, c) for n, _, c in S.mlp_segments(64, 16)]
    assert a == b


def _pack(named, shapes):
    return np.concatenate([np.asarray(named[n], dtype=np.float64).reshape(-1) for n, _ in shapes])


def _identity_towers(d=2):
    P = {}
    for t in "hel":
        P[f"rms_{t}"] = np.ones(d)
        P[f"W_{t}"] = np.eye(d)
        P[f"b_{t}"] = np.zeros(d)
    return P


def test_worked_example_g1_interaction_and_fusion():
    """Hand-worked closed form G1 (tests/golden/recall_head_worked.txt)."""
    d = dt = 2
    P = _identity_towers()
    Wf = np.zeros((2, 18))
    Wf[0, 9] = 1.0
    Wf[1, 12] = 1.0
    Wf[1, 17] = -1.0
    P.update(W_f=Wf, b_f=np.zeros(2))
    rng = np.random.default_rng(1)
    for k in (1, 2):
        P.update({f"rms_{k}": np.ones(2), f"W_gate_{k}": rng.standard_normal((4, 2)),
                  f"W_up_{k}": rng.standard_normal((4, 2)), f"W_down_{k}": np.zeros((2, 4))})
    P.update(rms_o=np.ones(2), w_o=np.array([1.0, 0.0]), b_o=np.array([0.25]))
    params = _pack(P, Gt.paper_head_shapes(d, dt))
    q = Gt.paper_head_score(params, d, dt, 0.0, np.array([[1.0, -1.0]]), np.array([[1.0, 1.0]]),
                            np.array([[-1.0, -1.0]]))
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    z = (2 * s1 - 0.5, 1.5 * s1 - 1.0)
    expect = z[0] / math.sqrt((z[0] ** 2 + z[1] ** 2) / 2) + 0.25
    assert q[0] == pytest.approx(expect, abs=1e-14)


def test_worked_example_g2_swiglu_block():
    """Hand-worked closed form G2 (tests/golden/recall_head_worked.txt)."""
    d = dt = 2
    P = _identity_towers()
    P.update(W_f=np.zeros((2, 18)), b_f=np.zeros(2))
    P.update(rms_1=np.ones(2), W_gate_1=np.array([[1, 0], [0, 1], [0, 0], [-1, -1]], float),
             W_up_1=np.array([[1, 0], [0, 0], [0, 1], [1, 1]], float),
             W_down_1=np.array([[1, 0, 0, 0], [0, 0, 0, 1]], float))
    P.update(rms_2=np.ones(2), W_gate_2=np.ones((4, 2)), W_up_2=np.ones((4, 2)), W_down_2=np.zeros((2, 4)))
    P.update(rms_o=np.ones(2), w_o=np.array([1.0, -1.0]), b_o=np.array([0.0]))
    params = _pack(P, Gt.paper_head_shapes(d, dt))
    one = np.array([[1.0, 1.0]])
    q = Gt.paper_head_score(params, d, dt, 0.0, one, one, one)
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    silu_m2 = -2.0 / (1.0 + math.exp(2.0))
    z1 = (2.5 * s1, 1.5 * s1 + 2 * silu_m2)
    expect = (z1[0] - z1[1]) / math.sqrt((z1[0] ** 2 + z1[1] ** 2) / 2)
    assert q[0] == pytest.approx(expect, abs=1e-14)


def _random_head(d, dt, seed=0):
    return S.gate_params(seed, "paper", d, dt).astype(np.float64)


def test_each_input_is_rms_normalised():
    """RMSNorm on every tower input: with eps = 0 the score is invariant to a
    positive rescaling of each input separately."""
    d, dt = 48, 8
    p = _random_head(d, dt)
    h, e, l = S.gate_inputs(2, 1, 3, d)
    h, e, l = (x[0].astype(np.float64) for x in (h, e, l))
    q0 = Gt.paper_head_score(p, d, dt, 0.0, h, e, l)
    for sh, se, sl in ((3.0, 1, 1), (1, 0.25, 1), (1, 1, 7.5)):
        q1 = Gt.paper_head_score(p, d, dt, 0.0, h * sh, e * se, l * sl)
        np.testing.assert_allclose(q1, q0, rtol=1e-12, atol=1e-12)
    # and not to a sign flip (SiLU is not odd)
    assert not np.allclose(Gt.paper_head_score(p, d, dt, 0.0, -h, e, l), q0)


def test_tower_swap_symmetry_of_interaction_vector():
    """Swapping the roles of the first two towers (inputs, weights) and
    permuting the fusion weight's column blocks to match leaves q unchanged:
    u's pairwise terms are symmetric (products and absolute differences)."""
    d, dt = 32, 8
    shapes = Gt.paper_head_shapes(d, dt)
    P = Gt.unpack(_random_head(d, dt, 4), shapes)
    h, e, l = (x[0] for x in S.gate_inputs(5, 1, 2, d))
    q0 = Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l)
    Q = dict(P)
    for nm in ("rms", "W", "b"):
        Q[f"{nm}_h"], Q[f"{nm}_e"] = P[f"{nm}_e"], P[f"{nm}_h"]
    blocks = [P["W_f"][:, i * dt:(i + 1) * dt] for i in range(9)]
    # under a <-> b:  [a;b;c;ab;|a-b|;ac;|a-c|;bc;|b-c|] -> [b;a;c;ab;|a-b|;bc;|b-c|;ac;|a-c|]
    perm = [1, 0, 2, 3, 4, 7, 8, 5, 6]
    Q["W_f"] = np.concatenate([blocks[perm[i]] for i in range(9)], axis=1)
    q1 = Gt.paper_head_score(_pack(Q, shapes), d, dt, 1e-6, e, h, l)
    np.testing.assert_allclose(q1, q0, rtol=1e-12, atol=1e-12)


def test_zero_down_projection_makes_block_identity():
    """P12 / residual: W_f = 0, b_f = 0 gives z0 = (a+b+c)/2; zero down
    projections leave z unchanged, so q depends on the towers only."""
    d, dt = 16, 4
    shapes = Gt.paper_head_shapes(d, dt)
    P = Gt.unpack(_random_head(d, dt, 9), shapes)
    P["W_f"][:] = 0
    P["b_f"][:] = 0
    P["W_down_1"][:] = 0
    P["W_down_2"][:] = 0
    h, e, l = (x[0] for x in S.gate_inputs(1, 1, 4, d))
    q = Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l)
    # changing any gate/up weight can no longer matter
    P["W_gate_1"] *= -3
    P["W_up_2"] += 1
    q2 = Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l)
    assert np.array_equal(q, q2)
    # but changing a tower does
    P["b_l"] += 0.5
    assert not np.allclose(Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l), q)


def test_output_bias_shifts_score():
    d, dt = 16, 4
    shapes = Gt.paper_head_shapes(d, dt)
    P = Gt.unpack(_random_head(d, dt, 2), shapes)
    h, e, l = (x[0] for x in S.gate_inputs(3, 1, 3, d))
    q0 = Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l)
    P["b_o"] = P["b_o"] + 0.375
    q1 = Gt.paper_head_score(_pack(P, shapes), d, dt, 1e-6, h, e, l)
    np.testing.assert_allclose(q1 - q0, 0.375, atol=1e-14)


def test_mlp_stand_in_matches_torch_layers():
    """P16: the stand-in is Linear -> exact GELU -> Linear (torch, fp64)."""
    d, hdim = 64, 16
    p = S.gate_params(6, "mlp", d, hdim).astype(np.float64)
    x = S.gate_inputs(6, 1, 5, d)[2][0].astype(np.float64)
    P = Gt.unpack(p, Gt.mlp_shapes(d, hdim))
    xt = torch.tensor(x)
    hid = torch.nn.functional.gelu(torch.nn.functional.linear(xt, torch.tensor(P["W1"]), torch.tensor(P["b1"])),
                                   approximate="none")
    ref = torch.nn.functional.linear(hid, torch.tensor(P["w2"])[None, :], torch.tensor(P["b2"]))[:, 0]
    np.testing.assert_allclose(Gt.mlp_score(p, d, hdim, x), ref.numpy(), rtol=1e-13, atol=1e-15)


def test_gelu_and_silu_special_values():
    assert Gt.gelu(np.array([0.0]))[0] == 0.0
    assert Gt.gelu(np.array([1.0]))[0] == pytest.approx(0.8413447460685429, abs=1e-15)   # Phi(1)
    assert Gt.silu(np.array([0.0]))[0] == 0.0
    assert Gt.silu(np.array([2.0]))[0] - Gt.silu(np.array([-2.0]))[0] == pytest.approx(2.0, abs=1e-15)


def test_decision_rule():
    """§2.1 / Alg. 1: Full iff q > theta (strict) or q nonfinite; a prescribed
    schedule still sends nonfinite scores to Full."""
    sc = np.array([0.0, 1e-9, -1e-9, np.nan, np.inf, -np.inf, 5.0])
    assert Gt.decide(sc, 0.0).tolist() == [False, True, False, True, True, True, True]
    assert Gt.decide(sc, np.inf).tolist() == [False, False, False, True, True, True, False]
    assert Gt.decide(sc, -np.inf).tolist() == [True, True, True, True, True, True, True]
    forced = np.array([0, 0, 1, 0, 0, 0, 0])
    assert Gt.decide(sc, 0.0, forced).tolist() == [False, False, True, True, True, True, False]
    w, n = Gt.compact(Gt.decide(sc, 0.0))
    assert w.tolist() == [1, 3, 4, 5, 6] and n == 5


@pytest.mark.parametrize("k,expected", [(2, 126), (4, 252), (8, 504)])
def test_runtime_schedule_counts(k, expected):
    """P14: the first 2/4/8 of every 16 steps over 1,008 routed steps give
    exactly 126/252/504 Full calls (App. B.7)."""
    sched = S.periodic_schedule(1008, k)
    flags = Gt.decide(np.zeros(1008), 0.0, forced=sched)
    assert int(flags.sum()) == expected
    sc = np.zeros(1008)
    sc[17] = np.nan          # a nonfinite score triggers Full and breaks the count
    assert int(Gt.decide(sc, 0.0, forced=sched).sum()) == expected + (0 if sched[17] else 1)
