"""One whole decode step on the GPU (Local -> gate -> Full for flagged
requests, in stream order on one stream) against the oracle's step, and the
step-level invariants: gate always-on selects Full everywhere (P2), gate
always-off leaves the Local result and Full writes nothing (P3)."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import FLAG_BORDER, AttnProblem, check_close, dev_f32
from oracle import step as OS

pytestmark = pytest.mark.gpu


def _step(p, g, gate_kind, d, dh, h, e, l, tau, s=4, W=24, forced=None):
    P = p.P
    B = p.B
    out, lse = p.new_out(np.nan)
    ws_l = torch.zeros(P.attn_workspace_size(p.shape, s, W), dtype=torch.uint8, device="cuda")
    ws_f = torch.zeros(P.attn_workspace_size(p.shape, 0, 0), dtype=torch.uint8, device="cuda")
    ws_g = torch.zeros(P.gate_workspace_size(g, B), dtype=torch.uint8, device="cuda")
    score = torch.empty(B, dtype=torch.float32, device="cuda")
    flags = torch.empty(B, dtype=torch.int32, device="cuda")
    wl = torch.empty(B, dtype=torch.int32, device="cuda")
    nw = torch.empty(1, dtype=torch.int32, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int64, device="cuda")
    dh_, de_, dl_ = dev_f32(h), dev_f32(e), dev_f32(l)
    fo = None if forced is None else torch.from_numpy(forced.astype(np.int32)).cuda()
    P.local_decode_attn(p.shape, p.inp, s, W, out, lse, ws_l)
    P.recall_gate(g, B, dh_, de_, dl_, tau, fo, score, flags, wl, nw, ctr, ws_g)
    P.full_decode_attn(p.shape, p.inp, 0, None, wl, nw, out, lse, ws_f)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy(), score.cpu().numpy(), flags.cpu().numpy(), int(ctr.item())


@pytest.mark.parametrize("gate_kind", ["paper", "mlp"])
@pytest.mark.parametrize("cur", [False, True])
def test_step_matches_oracle(gate_kind, cur):
    seq = [50, 90, 200, 3, 130, 64]
    B = len(seq)
    d, dh = 512, 64      # Hq * D == d_model, as in the measured configurations
    p = AttnProblem(21, 2, B, 8, 2, 64, seq, cur=cur, split_blocks=2)
    params = S.gate_params(5, gate_kind, d, dh)
    dp = dev_f32(params)
    g = p.P.gate_desc(p.P.HEAD_PAPER if gate_kind == "paper" else p.P.HEAD_MLP, d, dh, dp, 1e-6)
    h, e, l = (x[0] for x in S.gate_inputs(6, 1, B, d))
    ref0 = OS.decode_step(p.q, p.k, p.v, p.table, p.seq, p.scale, 4, 24, gate_kind, params, d, dh, 1e-6,
                          h.astype(np.float64), e.astype(np.float64), l.astype(np.float64), np.inf,
                          k_cur=p.kc, v_cur=p.vc)
    tau = float(np.median(ref0["score"]))
    tau = tau + (1e-3 if abs(tau) < 1 else 1e-3 * abs(tau))    # keep clear of the 1e-4 border
    ref = OS.decode_step(p.q, p.k, p.v, p.table, p.seq, p.scale, 4, 24, gate_kind, params, d, dh, 1e-6,
                         h.astype(np.float64), e.astype(np.float64), l.astype(np.float64), tau,
                         k_cur=p.kc, v_cur=p.vc)
    out, lse, score, flags, ctr = _step(p, g, gate_kind, d, dh, h, e, l, tau)
    assert not np.any(np.abs(ref["score"] - tau) < FLAG_BORDER)
    assert np.array_equal(flags, ref["flags"]) and ctr == ref["n_work"]
    assert 0 < ctr < B
    check_close(out, ref["out"])
    assert np.max(np.abs(lse - ref["lse"])) < 1e-4


def test_gate_always_on_gives_full_and_always_off_gives_local():
    seq = [77, 300, 1000]
    B = len(seq)
    d, dh = 4096, 256
    p = AttnProblem(31, 2, B, 32, 8, 128, seq)
    params = S.gate_params(2, "paper", d, dh)
    dp = dev_f32(params)
    g = p.P.gate_desc(p.P.HEAD_PAPER, d, dh, dp, 1e-6)
    h, e, l = (x[0] for x in S.gate_inputs(3, 1, B, d))
    loc = p.run_local(4, 24)
    full = p.run_full(0)
    out_on, _, _, flags_on, c_on = _step(p, g, "paper", d, dh, h, e, l, -np.inf)
    assert flags_on.tolist() == [1] * B and c_on == B
    assert np.array_equal(out_on, full[0].cpu().numpy())            # P2, bit-exact (same kernels)
    out_off, _, _, flags_off, c_off = _step(p, g, "paper", d, dh, h, e, l, np.inf)
    assert flags_off.tolist() == [0] * B and c_off == 0
    assert np.array_equal(out_off, loc[0].cpu().numpy())             # P3: Full wrote nothing
    ref_full = p.oracle_full(0)
    check_close(out_on, ref_full[0])
