"""Seeded random decode-attention problems against the fp64 oracle: layer
counts, batch, GQA group, head dimension, lengths, sinks, windows, split
sizes, candidate K/V, the Full selection mode, a native window for Full and
a length bound above the longest request all drawn per case.  One
zero-filled workspace serves every call of a case (Local, then Full over the
flags or the compacted list), so the in-launch split merge and its ticket
words are exercised across calls with different plans."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import AttnProblem, check_close, dev_i32

pytestmark = pytest.mark.gpu


def _case(seed):
    g = np.random.default_rng(1000 + seed)
    L = int(g.integers(1, 4))
    B = int(g.integers(1, 6))
    Hkv = int(g.choice([1, 2, 4]))
    G = int(g.choice([1, 2, 4, 8, 16]))
    D = int(g.choice([64, 128]))
    seq = g.integers(1, 601, size=B).tolist()
    s = int(g.integers(0, 21))
    w = int(g.integers(1, 701))
    split = int(g.choice([0, 0, 2, 4, 6, 8]))
    cur = bool(g.integers(0, 2))
    mode = str(g.choice(["flags", "list", "all"]))
    flags = (g.random(B) < 0.5).astype(np.int32)
    native = int(g.choice([0, 0, int(g.integers(1, 701))]))     # Full: whole history or a native window
    slack = int(g.choice([0, 0, int(g.integers(1, 200))]))      # max_seq_len above the longest request
    return L, B, Hkv * G, Hkv, D, seq, s, w, split, cur, mode, flags, native, slack


@pytest.mark.parametrize("seed", range(200))
def test_random_problems(seed):
    L, B, Hq, Hkv, D, seq, s, w, split, cur, mode, flags, native, slack = _case(seed)
    pb = AttnProblem(2000 + seed, L, B, Hq, Hkv, D, seq, cur=cur, split_blocks=split, max_len=max(seq) + slack)
    P = pb.P
    ws = torch.zeros(max(256, P.attn_workspace_size(pb.shape, s, w), P.attn_workspace_size(pb.shape, 0, native)),
                     dtype=torch.uint8, device="cuda")
    out, lse = pb.new_out(np.nan)
    P.local_decode_attn(pb.shape, pb.inp, s, w, out, lse, ws)
    torch.cuda.synchronize()
    want, want_lse, _ = pb.oracle_local(s, w)
    check_close(out.cpu().numpy(), want, what=f"local case {seed}")
    assert np.abs(lse.cpu().numpy() - want_lse).max() < 1e-4

    sel = list(range(B)) if mode == "all" else np.flatnonzero(flags).tolist()
    fl = dev_i32(flags) if mode == "flags" else None
    wl = dev_i32(sel + [0] * (B - len(sel))) if mode == "list" else None
    nw = dev_i32([len(sel)]) if mode == "list" else None
    P.full_decode_attn(pb.shape, pb.inp, native, fl, wl, nw, out, lse, ws)
    torch.cuda.synchronize()
    full, full_lse, _ = pb.oracle_full(native)
    o, ls = out.cpu().numpy(), lse.cpu().numpy()
    for b in range(B):
        ref, ref_lse = (full, full_lse) if b in sel else (want, want_lse)
        check_close(o[:, b], ref[:, b], what=f"case {seed} request {b} ({mode})")
        assert np.abs(ls[:, b] - ref_lse[:, b]).max() < 1e-4
    units = L * B * Hkv
    assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0
