"""Parity at the measured configurations' full sizes, in the launch
configuration bench.py times (stacked calls, automatic work plan, Local from
the direct-ring workspace; the Mixed step also with Local from the paged
cache): one decode step on the GPU, then sampled (layer, request) rows
recomputed by the fp64 oracle from copies of exactly the blocks those rows
read.  Gate scores and flags are compared for every request."""
import gc
import math

import numpy as np
import pytest
import torch

from harness import FLAG_BORDER, check_close, note_flags
from oracle import attention as OA
from oracle import gate as OG

pytestmark = pytest.mark.gpu


def _bench(name, head="paper", local="ring"):
    import bench as BN
    from paper_2609_20734_amd import workloads as WL
    return BN.Bench(WL.ALL[name], head, 1234, 1, local=local)


def _host_slice(b, st, layer, req):
    """Host copies of one request's blocks of one layer, with a renumbered table."""
    n = int(b.seq_host[req])
    nblk = (n + 15) // 16
    phys = b.dtable[req, :nblk].long()
    k = st.k[layer].index_select(0, phys).cpu().view(torch.int16).numpy().view(np.uint16)[None]
    v = st.v[layer].index_select(0, phys).cpu().view(torch.int16).numpy().view(np.uint16)[None]
    q = st.q[layer:layer + 1, req:req + 1].cpu().numpy().view(np.uint16)
    table = np.arange(nblk, dtype=np.int32)[None, :]
    return q, k, v, table, np.array([n], dtype=np.int32)


def _run_step(b, tau):
    calls = b.step_calls(tau)[0]
    for c in calls:
        c()
    torch.cuda.synchronize()


def _check_gate(b, tau):
    wl = b.wl
    params = b.params.cpu().numpy()
    h, e, l = (x[0].cpu().numpy().astype(np.float64) for x in (b.h, b.e, b.l))
    if b.head == "paper":
        ref = OG.paper_head_score(params, wl.d_model, wl.d_hidden, 1e-6, h, e, l)
    else:
        ref = OG.mlp_score(params, wl.d_model, wl.d_hidden, l)
    sc = b.score.cpu().numpy()
    assert np.max(np.abs(sc - ref)) <= 1e-4 * max(1.0, float(np.max(np.abs(ref))))
    flags = b.flags.cpu().numpy().astype(bool)
    want = OG.decide(ref, tau)
    border = np.abs(ref - tau) < FLAG_BORDER
    note_flags(f"full-size {wl.name} {b.head} head tau={tau:.6g}", border, flags != want)
    assert not np.any((flags != want) & ~border)
    n = int(b.n_work.item())
    assert n == int(flags.sum()) and np.array_equal(b.work.cpu().numpy()[:n], np.flatnonzero(flags))
    return flags


def _check_rows(b, flags, samples):
    for si, layer, req in samples:
        st = b.stacks[si]
        q, k, v, table, seq = _host_slice(b, st, layer, req)
        if flags[req]:
            f = lambda n: OA.native_window_set(n, st.stack.native_window)
        elif st.stack.gated:
            f = lambda n: OA.local_set(n, st.stack.local_sink, st.stack.local_window)
        else:
            f = lambda n: OA.native_window_set(n, st.stack.native_window)
        ref, lse_ref, _ = OA.decode_attention(q, k, v, table, seq, f, 1.0 / math.sqrt(b.wl.head_dim))
        got = st.out[layer, req].cpu().numpy()
        check_close(got, ref[0, 0], what=f"{st.stack.name} layer {layer} request {req}")
        assert np.max(np.abs(st.lse[layer, req].cpu().numpy() - lse_ref[0, 0])) < 1e-4


def _median_tau(b):
    sc = b.scores()[0]
    s = np.sort(sc)
    if len(s) == 1:
        return None
    m = len(s) // 2
    return float(0.5 * (s[m - 1] + s[m]))


@pytest.fixture(autouse=True)
def _release_memory():
    yield
    gc.collect()
    torch.cuda.empty_cache()


def test_llama_full_size():
    b = _bench("llama3-8b")
    for tau in (math.inf, -math.inf):
        _run_step(b, tau)
        flags = _check_gate(b, tau)
        _check_rows(b, flags, [(0, 0, 0), (0, 16, 0), (0, 31, 0)])


def _sampled_requests(b, flags, k, seed):
    """k seeded requests, always including a flagged and an unflagged one."""
    rng = np.random.default_rng(seed)
    on, off = np.flatnonzero(flags), np.flatnonzero(~flags)
    pick = {int(on[0]), int(off[0])} if len(on) and len(off) else set()
    for r in rng.permutation(b.wl.batch):
        if len(pick) >= k:
            break
        pick.add(int(r))
    return sorted(pick)


def test_long_full_size():
    """Layers {0, L/2, L-1} x every request (the four 131,072-position ones)."""
    b = _bench("long")
    tau = _median_tau(b)
    _run_step(b, tau)
    flags = _check_gate(b, tau)
    assert 0 < flags.sum() < b.wl.batch
    _check_rows(b, flags, [(0, l, r) for l in (0, 16, 31) for r in range(b.wl.batch)])


@pytest.mark.parametrize("local", ["ring", "paged"])
def test_mixed_full_size(local):
    """Layers {0, L/2, L-1} x four seeded requests, plus the longest flagged
    and the shortest unflagged request."""
    b = _bench("mixed", local=local)
    tau = _median_tau(b)
    _run_step(b, tau)
    flags = _check_gate(b, tau)
    on = np.flatnonzero(flags)
    off = np.flatnonzero(~flags)
    lens = b.seq_host
    longest_on = int(on[np.argmax(lens[on])])
    shortest_off = int(off[np.argmin(lens[off])])
    reqs = _sampled_requests(b, flags, 4, 7)
    _check_rows(b, flags, [(0, l, r) for l in (0, 16, 31) for r in reqs]
                + [(0, 5, longest_on), (0, 27, shortest_off)])


def test_hybrid_full_size():
    """Both layer groups (stack 0: native sliding-window layers; stack 1:
    global, ODA-gated layers) at their first, middle and last layer x four
    seeded requests."""
    b = _bench("hybrid")
    tau = _median_tau(b)
    _run_step(b, tau)
    flags = _check_gate(b, tau)
    reqs = _sampled_requests(b, flags, 4, 8)
    rows = []
    for si, st in enumerate(b.stacks):
        L = st.stack.num_layers
        rows += [(si, l, r) for l in (0, L // 2, L - 1) for r in reqs]
    _check_rows(b, flags, rows)


def test_hybrid_full_size_one_request_flagged():
    """One request flagged by a prescribed schedule: the gated layers' Full
    launch covers the request's 96 (layer, KV head) units in 5 splits each
    (480 workgroups, about two per CU) merged in the launch, the natively
    windowed layers' in one split each."""
    b = _bench("hybrid")
    B = b.wl.batch
    forced = torch.zeros((1, B), dtype=torch.int32, device="cuda")
    forced[0, 5] = 1
    for c in b.step_calls(math.inf, forced)[0]:
        c()
    torch.cuda.synchronize()
    flags = b.flags.cpu().numpy().astype(bool)
    assert flags.tolist() == [r == 5 for r in range(B)]
    assert int(b.n_work.item()) == 1 and int(b.work[0].item()) == 5
    _check_rows(b, flags, [(1, 0, 5), (1, 6, 5), (1, 11, 5), (0, 0, 5), (0, 35, 5), (1, 4, 2), (0, 17, 7)])


def test_llama_per_layer_launches_eager_and_graph():
    """The per-layer launch mode (one call per layer, the gate reading staged
    inputs): parity with the oracle, and a captured graph of it replays to the
    eager result bit for bit."""
    b = _bench("llama3-8b")
    st = b.stacks[0]
    b.h_stage.copy_(b.h[0])
    b.e_stage.copy_(b.e[0])
    b.l_stage.copy_(b.l[0])
    for tau in (math.inf, -math.inf):
        for c in b.per_layer_calls(tau, None):
            c()
        torch.cuda.synchronize()
        flags = _check_gate(b, tau)
        _check_rows(b, flags, [(0, 0, 0), (0, 19, 0), (0, 31, 0)])
    eager = st.out.clone(), st.lse.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for c in b.per_layer_calls(-math.inf, None):
            c()
    for _ in range(3):
        st.out.fill_(0.0)
        st.lse.fill_(0.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.out, eager[0]) and torch.equal(st.lse, eager[1])
    del g


def test_hybrid_retry_on_gated_layers_only():
    """The gated-only retry variant: the natively windowed layers keep their
    (already native) Local result, the gated layers of flagged requests get
    Full."""
    b = _bench("hybrid")
    tau = _median_tau(b)
    for c in b.step_calls(tau, gated_only=True)[0]:
        c()
    torch.cuda.synchronize()
    flags = _check_gate(b, tau)
    on = int(np.flatnonzero(flags)[0])
    off = int(np.flatnonzero(~flags)[0])
    _check_rows(b, flags, [(0, 3, on), (0, 20, off), (1, 2, on), (1, 7, off)])


def test_hybrid_per_layer_launches():
    """Per-layer launches over both layer groups (natively windowed layers and
    gated global layers, one call per layer each) against the oracle."""
    b = _bench("hybrid")
    tau = _median_tau(b)
    b.h_stage.copy_(b.h[0])
    b.e_stage.copy_(b.e[0])
    b.l_stage.copy_(b.l[0])
    for c in b.per_layer_calls(tau, None):
        c()
    torch.cuda.synchronize()
    flags = _check_gate(b, tau)
    reqs = _sampled_requests(b, flags, 3, 9)
    rows = []
    for si, st in enumerate(b.stacks):
        L = st.stack.num_layers
        rows += [(si, l, r) for l in (1, L - 2) for r in reqs]
    _check_rows(b, flags, rows)
