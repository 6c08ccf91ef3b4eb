"""GPU parity of oda_local_decode_attn / oda_full_decode_attn against the
fp64 oracle, element by element."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import LSE_ABS, AttnProblem, check_close, dev_i32
from oracle import attention as OA

pytestmark = pytest.mark.gpu


def _cmp(prob, got, ref, requests=None):
    out, lse = got
    o_ref, l_ref, _ = ref
    o = out.cpu().numpy()
    l = lse.cpu().numpy()
    reqs = range(prob.B) if requests is None else requests
    for b in reqs:
        check_close(o[:, b], o_ref[:, b], what=f"out[:, {b}]")
        assert np.max(np.abs(l[:, b] - l_ref[:, b])) <= LSE_ABS


def test_tiny_config_local_and_full():
    """Tiny: 1 layer, 8q/2kv heads, D=64, n=1024, W=128, contiguous KV."""
    p = AttnProblem(1234, 1, 1, 8, 2, 64, [1024], permute=False)
    _cmp(p, p.run_local(4, 128), p.oracle_local(4, 128))
    _cmp(p, p.run_full(0), p.oracle_full(0))


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
def test_shapes_and_gqa_groups(D, G):
    Hkv = 2
    p = AttnProblem(10 + G + D, 2, 3, Hkv * G, Hkv, D, [1, 45, 333], permute=True, split_blocks=4)
    _cmp(p, p.run_local(4, 37), p.oracle_local(4, 37))
    _cmp(p, p.run_full(0), p.oracle_full(0))


@pytest.mark.parametrize("cur", [False, True])
@pytest.mark.parametrize("split_blocks", [2, 6, 0])
def test_boundary_lengths(cur, split_blocks):
    """n at every boundary of the access set: 1, s, s+1, W-1, W, W+1, s+W, s+W+1,
    partial first/last blocks, with the current token from the cache or k_cur."""
    s, W = 4, 40
    seq = [1, s, s + 1, W - 1, W, W + 1, s + W, s + W + 1, 16, 17, 63, 64, 65, 200]
    p = AttnProblem(77, 2, len(seq), 8, 2, 128, seq, cur=cur, split_blocks=split_blocks)
    _cmp(p, p.run_local(s, W), p.oracle_local(s, W))
    _cmp(p, p.run_local(0, W), p.oracle_local(0, W))
    _cmp(p, p.run_full(0), p.oracle_full(0))
    _cmp(p, p.run_full(W), p.oracle_full(W))


@pytest.mark.parametrize("s", [0, 1, 4, 16, 19, 33])
def test_sink_counts_and_shared_block(s):
    """Sinks spanning one or several blocks, and a block shared by the sink and
    the recent part."""
    seq = [20, 40, 50, 70, 100, 300]
    p = AttnProblem(5 + s, 1, len(seq), 4, 1, 64, seq, split_blocks=2)
    for W in (1, 8, 30, 64):
        _cmp(p, p.run_local(s, W), p.oracle_local(s, W))


def test_local_equals_full_when_window_covers_context():
    """P1 on the GPU: s + W >= n gives the same set; the two calls agree within
    fp32 rounding (different split plans) and both match the oracle."""
    seq = [1, 30, 200, 257]
    p = AttnProblem(3, 2, len(seq), 16, 4, 128, seq)
    loc = p.run_local(4, 260)
    full = p.run_full(0)
    np.testing.assert_allclose(loc[0].cpu().numpy(), full[0].cpu().numpy(), atol=2e-6, rtol=0)
    _cmp(p, loc, p.oracle_full(0))


@pytest.mark.parametrize("mode", ["flags", "list"])
def test_full_touches_only_selected_requests(mode):
    seq = [100, 37, 260, 5, 99]
    p = AttnProblem(9, 2, len(seq), 8, 2, 64, seq, split_blocks=2)
    sel = np.array([0, 1, 1, 0, 1], dtype=np.int32)
    out, lse = p.new_out(-7.0)
    if mode == "flags":
        p.run_full(0, flags=dev_i32(sel), out=out, lse=lse)
    else:
        wl = np.zeros(len(seq), np.int32)
        idx = np.flatnonzero(sel)
        wl[:len(idx)] = idx
        wl[len(idx):] = 0   # entries past n_work are never read as requests
        p.run_full(0, work_list=dev_i32(wl), n_work=dev_i32([len(idx)]), out=out, lse=lse)
    o = out.cpu().numpy()
    ref = p.oracle_full(0, requests=list(np.flatnonzero(sel)))
    for b in range(len(seq)):
        if sel[b]:
            check_close(o[:, b], ref[0][:, b])
        else:
            assert np.all(o[:, b] == -7.0) and np.all(lse.cpu().numpy()[:, b] == -7.0)


@pytest.mark.parametrize("mode", ["flags", "list"])
def test_few_selected_of_a_wide_batch(mode):
    """A few selected requests of a 70-request batch (two 64-wide flag words),
    one layer, automatic splits: the selected requests get several splits each
    and the grid's leading workgroups map to them by rank (ascending ids for
    flags, list order for a work list, here not ascending)."""
    g = np.random.default_rng(70)
    seq = g.integers(1, 400, size=70)
    pick = [69, 3, 64]
    seq[pick] = [1999, 1500, 777]
    p = AttnProblem(70, 1, 70, 8, 2, 64, seq.tolist())
    out, lse = p.new_out(-7.0)
    if mode == "flags":
        fl = np.zeros(70, np.int32)
        fl[pick] = 1
        p.run_full(0, flags=dev_i32(fl), out=out, lse=lse)
    else:
        wl = np.zeros(70, np.int32)
        wl[:3] = pick
        p.run_full(0, work_list=dev_i32(wl), n_work=dev_i32([3]), out=out, lse=lse)
    o, ls = out.cpu().numpy(), lse.cpu().numpy()
    ref = p.oracle_full(0, requests=pick)
    for b in range(70):
        if b in pick:
            check_close(o[:, b], ref[0][:, b], what=f"request {b}")
            assert np.max(np.abs(ls[:, b] - ref[1][:, b])) <= LSE_ABS
        else:
            assert np.all(o[:, b] == -7.0) and np.all(ls[:, b] == -7.0)


@pytest.mark.parametrize("L,B,Hkv,cur", [(4, 64, 8, False), (6, 16, 8, True), (8, 32, 8, False), (3, 40, 8, True)])
def test_local_layer_groups(L, B, Hkv, cur):
    """Batched Local with enough units that one work item walks several
    layers of a (request, KV head) in turn (4, 3, 8 and 3 layers here): every
    layer's rows against the oracle, including a request whose length is out
    of range (NaN rows in every layer of its groups)."""
    g = np.random.default_rng(L * 100 + B)
    seq = g.integers(1, 300, size=B)
    seq[3] = 290
    p = AttnProblem(L * 100 + B, L, B, Hkv, Hkv, 64, seq.tolist(), cur=cur)
    bad = p.seq.copy()
    bad[5] = 0                                   # outside [1, max_seq_len]
    p.dseq = dev_i32(bad)
    p.inp = p.P.inputs(p.dq, p.dk, p.dv, p.dtable, p.dseq, p.scale, p.dkc, p.dvc)
    out, lse = p.run_local(4, 96)
    o, ls = out.cpu().numpy(), lse.cpu().numpy()
    ref, ref_lse, _ = p.oracle_local(4, 96, requests=[b for b in range(B) if b != 5])
    for b in range(B):
        if b == 5:
            assert np.isnan(o[:, b]).all() and np.isnan(ls[:, b]).all()
            continue
        check_close(o[:, b], ref[:, b], what=f"request {b}")
        assert np.max(np.abs(ls[:, b] - ref_lse[:, b])) <= LSE_ABS


def test_empty_work_list_writes_nothing():
    p = AttnProblem(2, 1, 3, 8, 2, 64, [10, 20, 30])
    out, lse = p.new_out(3.5)
    p.run_full(0, work_list=dev_i32([0, 0, 0]), n_work=dev_i32([0]), out=out, lse=lse)
    assert torch.all(out == 3.5) and torch.all(lse == 3.5)


def test_reruns_are_bit_identical():
    seq = [333, 1000]
    p = AttnProblem(4, 2, 2, 32, 8, 128, seq)
    a = p.run_local(4, 256)
    b = p.run_local(4, 256)
    c = p.run_full(0)
    d = p.run_full(0)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    assert torch.equal(c[0], d[0]) and torch.equal(c[1], d[1])


@pytest.mark.parametrize("n,s,W", [(300, 4, 64), (300, 0, 64), (70, 4, 66), (129, 19, 50)])
def test_dominant_key_probes(n, s, W):
    """P10 on the GPU: a key aligned with q at position p dominates iff p is in
    the access set, so out ~ V_p exactly at the set's boundaries."""
    p = AttnProblem(8, 1, 1, 1, 1, 64, [n], split_blocks=2)
    p.q[:] = S.f32_to_bf16_bits(np.float32(1.0))
    p.k = S.f32_to_bf16_bits(S.bf16_bits_to_f32(p.k) * np.float32(0.05))
    members = set(OA.local_set(n, s, W).tolist())
    for pos in sorted({0, s - 1, s, n - W - 1, n - W, n - 1}):
        if not (0 <= pos < n):
            continue
        k = p.k.copy()
        k[0, p.table[0][pos // 16], 0, :, pos % 16, :] = S.f32_to_bf16_bits(np.float32(8.0))
        saved = p.k
        p.k = k
        p.upload()
        out, _ = p.run_local(s, W)
        ref = p.oracle_local(s, W)
        check_close(out.cpu().numpy(), ref[0])
        vp = OA.bf16_to_f64(p.v[0, p.table[0][pos // 16], 0, :, pos % 16])
        hit = np.max(np.abs(out.cpu().numpy()[0, 0, 0] - vp)) < 1e-5
        assert hit == (pos in members), (pos, hit)
        p.k = saved
    p.upload()


def test_nan_in_unattended_slots_is_ignored():
    """Slots outside the access set may hold anything; NaN there must not leak."""
    seq = [40, 23]
    p = AttnProblem(6, 1, 2, 8, 2, 128, seq, split_blocks=2)
    nanbits = np.uint16(0x7FC0)
    for b, n in enumerate(seq):
        for pos in range(n, ((n + 15) // 16) * 16):       # tail of the last block
            p.k[:, p.table[b][pos // 16], :, :, pos % 16, :] = nanbits
            p.v[:, p.table[b][pos // 16], :, :, pos % 16] = nanbits
        for pos in range(4, 16):                          # between sinks and window
            if pos < n - 8:
                p.k[:, p.table[b][0], :, :, pos, :] = nanbits
                p.v[:, p.table[b][0], :, :, pos] = nanbits
    p.upload()
    _cmp(p, p.run_local(4, 8), p.oracle_local(4, 8))


@pytest.mark.parametrize("cur", [False, True])
def test_one_workspace_serves_many_calls(cur):
    """Split-K partials are merged by the last split of each request in the
    same launch, counting with ticket words at the front of the workspace.
    One zero-filled workspace, reused by Local and Full calls with different
    windows and selections, gives results bit-identical to fresh workspaces,
    matches the oracle, and is left with every ticket word zero."""
    pb = AttnProblem(41, 3, 4, 16, 4, 64, [300, 77, 513, 160], cur=cur, split_blocks=2)
    P = pb.P
    sizes = [P.attn_workspace_size(pb.shape, s, w) for s, w in ((4, 64), (0, 32), (0, 0))]
    ws = torch.zeros(max(sizes), dtype=torch.uint8, device="cuda")
    wl, nw = dev_i32([3, 0, 2, 1]), dev_i32([3])
    calls = [("local", 4, 64, None), ("full", 0, 0, None), ("local", 0, 32, None), ("full", 0, 0, (wl, nw)),
             ("local", 4, 64, None)]
    for kind, s, w, sel in calls:
        out, lse = pb.new_out(7.0)
        ref_out, ref_lse = pb.new_out(7.0)
        if kind == "local":
            P.local_decode_attn(pb.shape, pb.inp, s, w, out, lse, ws)
            pb.run_local(s, w, ref_out, ref_lse)
            want = pb.oracle_local(s, w)
        else:
            args = (None, *sel) if sel else (None, None, None)
            P.full_decode_attn(pb.shape, pb.inp, 0, *args, out, lse, ws)
            pb.run_full(0, *args, out=ref_out, lse=ref_lse)
            want = pb.oracle_full(requests=[3, 0, 2] if sel else None)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
        rows = [3, 0, 2] if sel else range(pb.B)
        o = out.cpu().numpy()
        check_close(o[:, rows], want[0][:, rows])
        if sel:
            assert np.all(o[:, 1] == 7.0)
        units = pb.L * pb.B * pb.Hkv
        assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0


def test_repeated_list_entry_leaves_the_workspace_valid():
    """A work list that names a request twice (a caller bug the gate never
    produces) gives that request unspecified rows, but its merge tickets count
    modulo the split count, so they return to zero: the other listed request
    is correct, an unlisted one is untouched, and a normal call on the same
    workspace afterwards matches the oracle."""
    pb = AttnProblem(43, 2, 3, 8, 2, 128, [400, 230, 515], split_blocks=2)
    P = pb.P
    ws = torch.zeros(P.attn_workspace_size(pb.shape, 0, 0), dtype=torch.uint8, device="cuda")
    units = pb.L * pb.B * pb.Hkv
    out, lse = pb.new_out(7.0)
    P.full_decode_attn(pb.shape, pb.inp, 0, None, dev_i32([2, 2, 0]), dev_i32([3]), out, lse, ws)
    torch.cuda.synchronize()
    assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0
    o = out.cpu().numpy()
    check_close(o[:, [0]], pb.oracle_full(requests=[0])[0][:, [0]])
    assert np.all(o[:, 1] == 7.0)
    out, lse = pb.new_out(7.0)
    P.full_decode_attn(pb.shape, pb.inp, 0, None, dev_i32([1, 2]), dev_i32([2]), out, lse, ws)
    torch.cuda.synchronize()
    want = pb.oracle_full(requests=[1, 2])
    _cmp(pb, (out, lse), want, requests=[1, 2])
    assert np.all(out.cpu().numpy()[:, 0] == 7.0)
    assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0


@pytest.mark.parametrize("cur", [False, True])
def test_selection_sizes_on_one_workspace(cur):
    """Full calls over device-side selections of 0, 1, 5, 11 and 12 of 12
    requests (4 layers, 8 KV heads: 384 units, automatic and forced split-K)
    and a flags selection, on one workspace: each matches the oracle on the
    selected rows, leaves the others untouched, and leaves the ticket words
    zero."""
    g = np.random.default_rng(91)
    seq = g.integers(1, 900, size=12)
    seq[[2, 7]] = [1, 2000]
    for split_blocks in (0, 4):
        pb = AttnProblem(91 + split_blocks, 4, 12, 32, 8, 64, seq.tolist(), cur=cur, split_blocks=split_blocks)
        P = pb.P
        ws = torch.zeros(max(256, P.attn_workspace_size(pb.shape, 0, 0)), dtype=torch.uint8, device="cuda")
        units = pb.L * pb.B * pb.Hkv
        for sel in ([], [7], [11, 0, 2, 7, 5], [b for b in range(12) if b != 4], list(range(12)), "flags"):
            out, lse = pb.new_out(-7.0)
            if sel == "flags":
                fl = (np.arange(12) % 3 == 1).astype(np.int32)
                rows = list(np.flatnonzero(fl))
                P.full_decode_attn(pb.shape, pb.inp, 0, dev_i32(fl), None, None, out, lse, ws)
            else:
                rows = sel
                wl = np.zeros(12, np.int32)
                wl[:len(sel)] = sel
                P.full_decode_attn(pb.shape, pb.inp, 0, None, dev_i32(wl), dev_i32([len(sel)]), out, lse, ws)
            torch.cuda.synchronize()
            assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0, (split_blocks, sel)
            o, ls = out.cpu().numpy(), lse.cpu().numpy()
            if rows:
                ref = pb.oracle_full(0, requests=rows)
                for b in rows:
                    check_close(o[:, b], ref[0][:, b], what=f"split {split_blocks} sel {sel} request {b}")
                    assert np.max(np.abs(ls[:, b] - ref[1][:, b])) <= LSE_ABS
            for b in set(range(12)) - set(rows):
                assert np.all(o[:, b] == -7.0) and np.all(ls[:, b] == -7.0)


def test_selection_sizes_with_balanced_splits():
    """96 (layer, KV head) units per request (12 layers x 8 KV heads) and a
    41,000-position history (2,563 blocks): Full over 1, 2, 3 and 4 selected
    requests takes 5, 4, 5 and 2 splits per unit, the counts that spread the
    workgroups evenly over the CUs, and merges them in the launch; the shorter
    requests get fewer splits.  Every selection on one workspace matches the
    oracle, leaves the unselected rows untouched and the ticket words zero."""
    seq = [41000, 3000, 1, 5000]
    pb = AttnProblem(97, 12, 4, 32, 8, 64, seq, cur=True)
    P = pb.P
    ws = torch.zeros(max(256, P.attn_workspace_size(pb.shape, 0, 0)), dtype=torch.uint8, device="cuda")
    units = pb.L * pb.B * pb.Hkv
    ref_o, ref_l, _ = pb.oracle_full(0, requests=[0, 1, 2, 3])
    for sel in ([0], [3, 0], [1, 0, 3], [2, 0, 3, 1]):
        out, lse = pb.new_out(-7.0)
        wl = np.zeros(4, np.int32)
        wl[:len(sel)] = sel
        P.full_decode_attn(pb.shape, pb.inp, 0, None, dev_i32(wl), dev_i32([len(sel)]), out, lse, ws)
        torch.cuda.synchronize()
        assert int(ws[:4 * units].view(torch.int32).abs().sum().item()) == 0, sel
        o, ls = out.cpu().numpy(), lse.cpu().numpy()
        for b in sel:
            check_close(o[:, b], ref_o[:, b], what=f"selection {sel} request {b}")
            assert np.max(np.abs(ls[:, b] - ref_l[:, b])) <= LSE_ABS
        for b in set(range(4)) - set(sel):
            assert np.all(o[:, b] == -7.0) and np.all(ls[:, b] == -7.0)


@pytest.mark.parametrize("cur,walk", [(False, False), (True, False), (True, True)])
def test_layer_stride_between_layers(cur, walk):
    """layer_stride_kv: each layer's blocks start `stride` elements after the
    previous layer's (here the dense size plus padding, as in one allocation
    holding several layer groups).  Local and Full read the right layers and
    match the oracle on the dense copies; `walk` takes a batch large enough
    that Local's workgroups each walk all four layers of a (request, KV head).
    Rings filled from the padded caches give Local the same bits."""
    if walk:
        seq = np.random.default_rng(58).integers(1, 300, size=64).tolist()
        pb = AttnProblem(58, 4, 64, 8, 8, 64, seq, cur=cur)
    else:
        pb = AttnProblem(57, 3, 4, 16, 4, 128, [70, 300, 1, 515], cur=cur, split_blocks=2)
    P = pb.P
    dense = pb.nb * pb.Hkv * 16 * pb.D
    stride = dense + 8 * 37
    k_pad = torch.zeros(pb.L * stride, dtype=torch.int16, device="cuda")
    v_pad = torch.zeros(pb.L * stride, dtype=torch.int16, device="cuda")
    for l in range(pb.L):
        k_pad[l * stride:l * stride + dense] = pb.dk[l].reshape(-1)
        v_pad[l * stride:l * stride + dense] = pb.dv[l].reshape(-1)
    shape = P.Shape(pb.L, pb.B, pb.Hq, pb.Hkv, pb.D, pb.shape.max_blocks_per_seq, pb.shape.max_seq_len, pb.nb,
                    pb.shape.split_blocks, layer_stride_kv=stride)
    inp = P.inputs(pb.dq, k_pad, v_pad, pb.dtable, pb.dseq, pb.scale, pb.dkc, pb.dvc)
    for local in (True, False):
        out, lse = pb.new_out(np.nan)
        ws = torch.zeros(max(256, P.attn_workspace_size(shape, 4, 64 if local else 0)), dtype=torch.uint8,
                         device="cuda")
        if local:
            P.local_decode_attn(shape, inp, 4, 64, out, lse, ws)
            want = pb.oracle_local(4, 64)
        else:
            P.full_decode_attn(shape, inp, 0, None, None, None, out, lse, ws)
            want = pb.oracle_full(0)
        torch.cuda.synchronize()
        _cmp(pb, (out, lse), want)
        if local:
            # rings filled from the padded layers give the same bits as the paged Local
            n = P.ring_elements(shape, 4, 64)
            kr = torch.full((n,), 0x7FC0, dtype=torch.int16, device="cuda")
            vr = torch.full((n,), 0x7FC0, dtype=torch.int16, device="cuda")
            P.ring_fill(shape, k_pad, v_pad, pb.dtable, pb.dseq, 4, 64, kr, vr)
            out_r, lse_r = pb.new_out(np.nan)
            P.local_decode_attn_ring(shape, P.inputs(pb.dq, None, None, None, pb.dseq, pb.scale, pb.dkc, pb.dvc),
                                     kr, vr, 4, 64, out_r, lse_r, ws)
            torch.cuda.synchronize()
            assert torch.equal(out_r.view(torch.int32), out.view(torch.int32))
            assert torch.equal(lse_r.view(torch.int32), lse.view(torch.int32))
