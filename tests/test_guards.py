"""Device data outside the ABI's contract (lengths outside [1, max_seq_len],
block-table entries outside [0, num_blocks), listed requests outside the
batch) is never used to address memory: the kernels' own checks turn it into
NaN rows or skipped requests, and every other request is computed exactly as
usual.  The bad values are written from the host; every kernel still reads
only valid addresses."""
import numpy as np
import pytest
import torch

import oda_synth as S
from harness import AttnProblem, check_close, dev_f32, dev_i32, dev_u16, need_gpu
from oracle import attention as OA

pytestmark = pytest.mark.gpu


def _rows_nan(x, b):
    return bool(np.isnan(x[:, b]).all())


@pytest.mark.parametrize("split_blocks", [0, 2])
@pytest.mark.parametrize("cur", [False, True])
def test_lengths_out_of_range_give_nan_rows(split_blocks, cur):
    pb = AttnProblem(31, 2, 4, 8, 2, 128, [20, 37, 70, 50], cur=cur, split_blocks=split_blocks)
    bad = pb.dseq.clone()
    bad[0] = 0
    bad[3] = 70 + 3                      # above the shape's max_seq_len
    pb.inp = pb.P.inputs(pb.dq, pb.dk, pb.dv, pb.dtable, bad, pb.scale, pb.dkc, pb.dvc)
    for run, ref in ((lambda: pb.run_local(4, 24), lambda: pb.oracle_local(4, 24, requests=[1, 2])),
                     (lambda: pb.run_full(), lambda: pb.oracle_full(requests=[1, 2]))):
        out, lse = (t.cpu().numpy() for t in run())
        want = ref()
        for b in (0, 3):
            assert _rows_nan(out, b) and _rows_nan(lse, b)
        check_close(out[:, [1, 2]], want[0][:, [1, 2]])


@pytest.mark.parametrize("split_blocks", [0, 2])
def test_table_entries_out_of_range_give_nan_rows(split_blocks):
    pb = AttnProblem(32, 2, 4, 8, 2, 128, [20, 37, 70, 50], split_blocks=split_blocks)
    tab = pb.dtable.clone()
    tab[1, 1] = pb.nb + 5               # request 1, logical block 1 (positions 16..31)
    tab[2, 0] = -1                      # request 2, logical block 0 (the sinks)
    pb.inp = pb.P.inputs(pb.dq, pb.dk, pb.dv, tab, pb.dseq, pb.scale)
    for run, ref in ((lambda: pb.run_local(4, 24), lambda: pb.oracle_local(4, 24, requests=[0, 3])),
                     (lambda: pb.run_full(), lambda: pb.oracle_full(requests=[0, 3]))):
        out, lse = (t.cpu().numpy() for t in run())
        want = ref()
        for b in (1, 2):
            assert _rows_nan(out, b) and _rows_nan(lse, b)
        check_close(out[:, [0, 3]], want[0][:, [0, 3]])


def test_listed_request_outside_the_batch_is_skipped():
    pb = AttnProblem(33, 2, 3, 8, 2, 64, [40, 17, 90])
    wl = dev_i32([2, 9, 0])
    nw = dev_i32([3])
    out, lse = pb.new_out(7.0)
    pb.run_full(work_list=wl, n_work=nw, out=out, lse=lse)
    o = out.cpu().numpy()
    want = pb.oracle_full(requests=[0, 2])
    check_close(o[:, [0, 2]], want[0][:, [0, 2]])
    assert np.all(o[:, 1] == 7.0)


def test_commit_writes_nothing_for_bad_lengths_or_entries():
    P = need_gpu()
    L, B, Hkv, D = 2, 4, 2, 64
    seq = np.array([5, 17, 40, 33], dtype=np.int32)
    table, nb = S.paged_block_table(S.rng(34, S.STREAM_TABLE), seq + 1, 4)
    k, v = S.kv_cache(34, L, nb, Hkv, D)
    kl = S.normal_bf16(S.rng(35, S.STREAM_KCUR), (L, B, Hkv, D))
    vl = S.normal_bf16(S.rng(35, S.STREAM_VCUR), (L, B, Hkv, D))
    dk, dv = dev_u16(k), dev_u16(v)
    tab = table.copy()
    tab[2, (40 - 1) // 16] = nb + 1      # request 2's slot block is out of range
    dseq = dev_i32([0, 17, 40, 4 * 16 + 1])   # request 0: length 0; request 3: beyond the table
    shape = P.Shape(L, B, 8, Hkv, D, 4, 64, nb)
    ws = torch.zeros(P.commit_workspace_size(shape), dtype=torch.uint8, device="cuda")
    P.commit_kv(shape, dk, dv, dev_i32(tab), dseq, dev_u16(kl), dev_u16(vl), workspace=ws)
    torch.cuda.synchronize()
    hk, hv = k.copy(), v.copy()
    pos = 16                              # request 1 (the only valid one) writes position 16
    blk = table[1, pos // 16]
    for l in range(L):
        for g in range(Hkv):
            hk[l, blk, g, :, pos % 16, :] = kl[l, 1, g].reshape(D // 8, 8)
            hv[l, blk, g, :, pos % 16] = vl[l, 1, g]
    assert np.array_equal(dk.cpu().numpy().view(np.uint16), hk)
    assert np.array_equal(dv.cpu().numpy().view(np.uint16), hv)
    assert dseq.cpu().numpy().tolist() == [1, 18, 41, 66]      # lengths still advance


def test_dense_and_row_copy_skip_listed_requests_outside_the_batch():
    P = need_gpu()
    g = S.rng(36, S.STREAM_DECODER)
    W = S.normal_bf16(g, (16, 64), 0.125)
    x = g.standard_normal((3, 64)).astype(np.float32)
    y = torch.full((3, 16), 7.0, device="cuda")
    P.dense_bf16(P.dense_desc(64, 16, P.DENSE_PLAIN, dev_u16(W)), 3, dev_f32(x), None, y, dev_i32([-1, 2, 5]),
                 dev_i32([3]))
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    ref = OA.bf16_to_f64(W) @ x[2].astype(np.float64)
    assert np.abs(got[2] - ref).max() <= 1e-4 * max(1.0, np.abs(ref).max())
    assert np.all(got[[0, 1]] == 7.0)
    dst = torch.full((3, 8), -1.0, device="cuda")
    src = dev_f32(np.arange(24, dtype=np.float32).reshape(3, 8))
    P.copy_rows(3, 8, src, dst, dev_i32([7, 1, -3]), dev_i32([3]))
    torch.cuda.synchronize()
    d = dst.cpu().numpy()
    assert np.all(d[1] == np.arange(8, 16)) and np.all(d[[0, 2]] == -1.0)


def test_stream_read_reads_and_leaves_the_sink():
    """The read-ceiling aid reads any 16-byte multiple and writes nothing
    (its sink keeps its value unless the XOR of the data hits one constant)."""
    P = need_gpu()
    x = torch.arange(1 << 20, dtype=torch.int32, device="cuda")
    sink = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    for nbytes, groups in ((x.numel() * 4, 0), (4096 + 16, 3), (16, 1), (x.numel() * 4, 1000)):
        P.stream_read(x, nbytes, sink, groups)
    torch.cuda.synchronize()
    assert int(sink.item()) == 12345
