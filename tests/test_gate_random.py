"""Seeded random recall-gate problems against the fp64 oracle: head kind,
model width, tower width, batch (ragged K chunks, tails, several batch
tiles), threshold and an optional prescribed schedule drawn per case; the
scores, flags, compacted list and recall counter are checked as in
test_gate_parity.py."""
import numpy as np
import pytest

import oda_synth as S
from oracle import gate as OG
from test_gate_parity import Gate, _check

pytestmark = pytest.mark.gpu


def _case(seed):
    g = np.random.default_rng(5000 + seed)
    kind = str(g.choice(["paper", "mlp"]))
    d = 4 * int(g.integers(1, 1100))
    dh = 4 * int(g.integers(1, 160 if kind == "paper" else 400))
    B = int(g.choice([1, 1, 2, 3, 5, 8, 9, 17, 33, 70]))
    forced = (g.random(B) < 0.3).astype(np.int32) if g.random() < 0.25 else None
    q = float(g.random())
    return kind, d, dh, B, forced, q


@pytest.mark.parametrize("seed", range(40))
def test_random_gates(seed):
    kind, d, dh, B, forced, q = _case(seed)
    gate = Gate(kind, d, dh, B, seed=100 + seed)
    h, e, l = (x[0] for x in S.gate_inputs(200 + seed, 1, B, d))
    ref = gate.oracle(h.astype(np.float64), e.astype(np.float64), l.astype(np.float64))
    tau = float(np.quantile(ref, q))
    _, fl, _ = _check(gate, h, e, l, tau, forced)
    assert int(gate.counter.item()) == int(fl.sum())
