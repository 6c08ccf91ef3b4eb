"""GPU parity of oda_recall_gate against the fp64 oracle: scores, flags
(bit-exact except where |score - tau| < 1e-4, counted), compaction, forced
schedules, nonfinite fallback and the recall counter."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import FLAG_BORDER, dev_f32, dev_i32, need_gpu, note_flags
from oracle import gate as OG

pytestmark = pytest.mark.gpu

SCORE_REL = 1e-4   # fp32 head vs fp64 oracle, relative to the score scale


class Gate:
    def __init__(self, kind, d, dh, batch, seed=1, eps=1e-6):
        self.P = need_gpu()
        self.kind, self.d, self.dh, self.B, self.eps = kind, d, dh, batch, eps
        self.params = S.gate_params(seed, kind, d, dh)
        assert self.params.size == self.P.gate_param_count(
            self.P.HEAD_PAPER if kind == "paper" else self.P.HEAD_MLP, d, dh)
        self.dparams = dev_f32(self.params)
        self.desc = self.P.gate_desc(self.P.HEAD_PAPER if kind == "paper" else self.P.HEAD_MLP, d, dh,
                                     self.dparams, eps)
        self.ws = torch.zeros(self.P.gate_workspace_size(self.desc, batch), dtype=torch.uint8, device="cuda")
        self.counter = torch.zeros(1, dtype=torch.int64, device="cuda")

    def run(self, h, e, l, tau, forced=None):
        B = self.B
        score = torch.full((B,), np.nan, dtype=torch.float32, device="cuda")
        flags = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        wl = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        nw = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        dh, de, dl = dev_f32(h), dev_f32(e), dev_f32(l)
        fo = dev_i32(forced) if forced is not None else None
        self.P.recall_gate(self.desc, B, dh, de, dl, tau, fo, score, flags, wl, nw, self.counter, self.ws)
        torch.cuda.synchronize()
        n = int(nw.item())
        return score.cpu().numpy(), flags.cpu().numpy(), wl.cpu().numpy()[:n], n

    def oracle(self, h, e, l):
        if self.kind == "paper":
            return OG.paper_head_score(self.params, self.d, self.dh, self.eps, h, e, l)
        return OG.mlp_score(self.params, self.d, self.dh, l)


def _check(g, h, e, l, tau, forced=None):
    sc, fl, wl, n = g.run(h, e, l, tau, forced)
    ref = g.oracle(h.astype(np.float64), e.astype(np.float64), l.astype(np.float64))
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(sc), fin)
    scale = max(1.0, float(np.max(np.abs(ref[fin]))) if fin.any() else 1.0)
    assert np.max(np.abs(sc[fin] - ref[fin]), initial=0.0) <= SCORE_REL * scale
    want = OG.decide(ref, tau, forced)
    border = fin & (np.abs(ref - tau) < FLAG_BORDER) & (forced is None)
    differ = fl.astype(bool) != want
    note_flags(f"gate {g.kind} d={g.d} dt={g.dh} B={g.B} tau={tau:.6g}", border, differ)
    mism = differ & ~border
    assert not mism.any(), np.flatnonzero(mism)
    # compaction: ascending flagged ids of the GPU's own flags, and its count
    assert n == int(fl.sum()) and np.array_equal(wl, np.flatnonzero(fl))
    return sc, fl, int(border.sum())


@pytest.mark.parametrize("kind,d,dh,B", [("mlp", 512, 64, 1), ("mlp", 512, 64, 13), ("paper", 512, 64, 1),
                                         ("paper", 64, 16, 9), ("paper", 4096, 256, 1), ("mlp", 4096, 256, 32),
                                         ("paper", 4096, 256, 32), ("paper", 8192, 512, 8),
                                         # launch shapes: K split over a workgroup, grouped rows, ragged
                                         # tiles and chunk tails, wide towers, batches over 64
                                         ("paper", 2048, 1024, 1), ("paper", 4096, 260, 70),
                                         ("paper", 256, 516, 2), ("mlp", 8192, 512, 8), ("mlp", 4096, 256, 70),
                                         # split-hidden SwiGLU blocks (one or two requests)
                                         ("paper", 1024, 128, 2), ("paper", 4096, 512, 1), ("paper", 256, 32, 2),
                                         # tower widths whose hidden units do not split into 1, 2 or 4 per
                                         # wavefront: unsplit blocks (these once ran the split kernel of
                                         # another width)
                                         ("paper", 1732, 192, 1), ("paper", 512, 384, 2), ("paper", 300, 96, 1),
                                         ("paper", 64, 12, 2),
                                         # 40 and 64 requests (several batch tiles), a few requests with short or
                                         # ragged rows
                                         ("paper", 1732, 192, 40), ("paper", 4096, 256, 64), ("paper", 100, 32, 4),
                                         ("paper", 4100, 64, 17)])
def test_scores_and_flags(kind, d, dh, B):
    g = Gate(kind, d, dh, B)
    h, e, l = (x[0] for x in S.gate_inputs(3, 1, B, d))
    ref = g.oracle(h.astype(np.float64), e.astype(np.float64), l.astype(np.float64))
    for tau in (float(np.median(ref)), 0.0, float(np.min(ref)) - 1, np.inf, -np.inf):
        _check(g, h, e, l, tau)


def test_tiny_threshold_recalls_5_of_16():
    """Tiny config: tau between the 5th and 6th largest of 16 scores -> 5/16."""
    g = Gate("mlp", 512, 64, 1)
    h, e, l = S.gate_inputs(1234, 16, 1, 512)
    ref = np.array([g.oracle(h[t].astype(np.float64), e[t].astype(np.float64), l[t].astype(np.float64))[0]
                    for t in range(16)])
    srt = np.sort(ref)[::-1]
    tau = float(0.5 * (srt[4] + srt[5]))
    total = 0
    for t in range(16):
        _, fl, _ = _check(g, h[t], e[t], l[t], tau)
        total += int(fl[0])
    assert total == 5
    assert int(g.counter.item()) == 5


def test_nonfinite_scores_go_to_full():
    """P13: NaN / Inf inputs give a nonfinite score -> flag 1, also when a
    prescribed schedule says Local."""
    B = 6
    for kind in ("paper", "mlp"):
        g = Gate(kind, 64, 16, B)
        h, e, l = (x[0].copy() for x in S.gate_inputs(4, 1, B, 64))
        l[1, 3] = np.nan
        l[4, 0] = np.inf
        sc, fl, wl, n = g.run(h, e, l, np.inf)
        assert not np.isfinite(sc[1]) and not np.isfinite(sc[4])
        assert fl.tolist() == [0, 1, 0, 0, 1, 0] and wl.tolist() == [1, 4]
        sc, fl, wl, n = g.run(h, e, l, np.inf, forced=np.array([1, 0, 0, 1, 0, 0], np.int32))
        assert fl.tolist() == [1, 1, 0, 1, 1, 0] and n == 4
    # the split-hidden blocks (two requests): NaN in one request stays in it
    g = Gate("paper", 256, 64, 2)
    h, e, l = (x[0].copy() for x in S.gate_inputs(5, 1, 2, 256))
    h[1, 7] = np.nan
    sc, fl, wl, n = g.run(h, e, l, np.inf)
    assert np.isfinite(sc[0]) and not np.isfinite(sc[1])
    assert fl.tolist() == [0, 1] and wl.tolist() == [1]


@pytest.mark.parametrize("k,expected", [(2, 126), (4, 252), (8, 504)])
def test_prescribed_schedule_counts(k, expected):
    """P14 on the device: the first k of every 16 steps over 1,008 routed steps
    -> exactly 126 / 252 / 504 Full calls, counted by the device counter."""
    g = Gate("mlp", 64, 16, 1)
    sched = S.periodic_schedule(1008, k)
    h, e, l = (x[:, 0] for x in S.gate_inputs(7, 1, 1, 64))
    score = torch.empty(1, dtype=torch.float32, device="cuda")
    flags = torch.empty(1, dtype=torch.int32, device="cuda")
    dh, de, dl = dev_f32(h), dev_f32(e), dev_f32(l)
    dsched = dev_i32(sched)
    for t in range(1008):
        g.P.recall_gate(g.desc, 1, dh, de, dl, 0.0, dsched[t:t + 1], score, flags, None, None, g.counter, g.ws)
    torch.cuda.synchronize()
    assert int(g.counter.item()) == expected


def test_equal_score_and_threshold_stays_local():
    """Strict '>': a score equal to the threshold keeps Local."""
    g = Gate("mlp", 64, 16, 4)
    h, e, l = (x[0] for x in S.gate_inputs(9, 1, 4, 64))
    sc, _, _, _ = g.run(h, e, l, 0.0)
    sc2, fl, _, _ = g.run(h, e, l, float(sc[2]))
    assert np.array_equal(sc, sc2)          # deterministic
    assert fl[2] == 0


def test_one_workspace_serves_heads_of_any_shape():
    """Every byte a gate call reads from its workspace it wrote earlier in the
    same call: one workspace, sized for the largest call and left holding the
    previous call's activations, serves heads of different batches, widths and
    launch paths in turn, each giving the results of a fresh workspace."""
    P = need_gpu()
    shapes = [("paper", 4096, 256, 32), ("paper", 4096, 256, 1), ("paper", 512, 64, 5), ("mlp", 4096, 256, 8),
              ("paper", 1024, 128, 64), ("paper", 4096, 256, 32)]
    gates = [Gate(kind, d, dh, B, seed=60 + i) for i, (kind, d, dh, B) in enumerate(shapes)]
    shared = torch.zeros(max(g.ws.numel() for g in gates), dtype=torch.uint8, device="cuda")
    for i, g in enumerate(gates):
        h, e, l = (x[0] for x in S.gate_inputs(70 + i, 1, g.B, g.d))
        fresh = g.run(h, e, l, 0.0)
        own = g.ws
        g.ws = shared
        again = g.run(h, e, l, 0.0)
        g.ws = own
        assert np.array_equal(fresh[0], again[0]) and np.array_equal(fresh[1], again[1]), shapes[i]
