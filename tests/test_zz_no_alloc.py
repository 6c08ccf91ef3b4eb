"""oda_recall_gate_static (the gate with the library's own static workspace,
for callers that cannot allocate) against oda_recall_gate with a caller
workspace: two calls in a row, the second with a smaller batch, and every
output -- scores, flags, the compacted list, its count and the recall
counter -- bit-identical (the same kernels run in the same order), and the
scores within the usual bar of the fp64 oracle."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import dev_f32, dev_i32, need_gpu
from oracle import gate as OG

pytestmark = pytest.mark.gpu


def _outputs(B):
    return (torch.full((B,), np.nan, dtype=torch.float32, device="cuda"),
            torch.full((B,), -1, dtype=torch.int32, device="cuda"),
            torch.full((B,), -1, dtype=torch.int32, device="cuda"),
            torch.full((1,), -1, dtype=torch.int32, device="cuda"),
            torch.zeros(1, dtype=torch.int64, device="cuda"))


@pytest.mark.parametrize("kind,d,dt,batches", [("paper", 4096, 256, (32, 1)), ("paper", 512, 64, (9, 2)),
                                               ("mlp", 4096, 256, (70, 3))])
def test_static_workspace_gate_matches_the_workspace_gate(kind, d, dt, batches):
    P = need_gpu()
    k = P.HEAD_PAPER if kind == "paper" else P.HEAD_MLP
    params = S.gate_params(21, kind, d, dt)
    desc = P.gate_desc(k, d, dt, dev_f32(params), 1e-6)
    for call, B in enumerate(batches):
        h, e, l = (x[0] for x in S.gate_inputs(30 + call, 1, B, d))
        dh, de, dl = dev_f32(h), dev_f32(e), dev_f32(l)
        if kind == "paper":
            ref = OG.paper_head_score(params, d, dt, 1e-6, h.astype(np.float64), e.astype(np.float64),
                                      l.astype(np.float64))
        else:
            ref = OG.mlp_score(params, d, dt, l.astype(np.float64))
        tau = float(np.median(ref))
        forced = dev_i32((np.arange(B) % 3 == 0).astype(np.int32)) if call == 1 else None
        a = _outputs(B)
        ws = torch.zeros(P.gate_workspace_size(desc, B), dtype=torch.uint8, device="cuda")
        P.recall_gate(desc, B, dh, de, dl, tau, forced, *a, ws)
        b = _outputs(B)
        P.recall_gate_static(desc, B, dh, de, dl, tau, forced, *b)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x, y), (call, B)
        sc = b[0].cpu().numpy()
        assert np.max(np.abs(sc - ref)) <= 1e-4 * max(1.0, float(np.max(np.abs(ref))))
        n = int(b[3].item())
        assert n == int(b[1].sum().item()) and int(b[4].item()) == n


def test_static_workspace_rejects_a_batch_beyond_its_size():
    P = need_gpu()
    params = torch.zeros(P.gate_param_count(P.HEAD_PAPER, 64, 1024), dtype=torch.float32, device="cuda")
    desc = P.gate_desc(P.HEAD_PAPER, 64, 1024, params, 1e-6)
    B = 600                                   # 28 * 600 * 1024 bytes > 16 MiB
    x = torch.zeros(B, 64, dtype=torch.float32, device="cuda")
    o = _outputs(B)
    with pytest.raises(P.OdaError) as err:
        P.recall_gate_static(desc, B, x, x, x, 0.0, None, *o)
    assert err.value.status == -4
    assert int(o[3].item()) == -1             # nothing was enqueued
