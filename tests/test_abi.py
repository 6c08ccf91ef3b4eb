"""The C-ABI library loads, exports every entry point include/oda.h declares,
and rejects bad arguments with the documented status codes before touching the
GPU (no device work is needed, so these run without one)."""
import ctypes
import math
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2609_20734_amd import build as B
    if not os.path.exists(B.LIB):
        B.build()
    import paper_2609_20734_amd._lib as lib
    return lib


def declared_functions():
    txt = open(os.path.join(ROOT, "include", "oda.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(oda_[a-z_0-9]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(L.EXPORTED), names
    for n in names:
        assert hasattr(L._lib, n), n


def _shape(L, **kw):
    base = dict(num_layers=2, batch=3, num_q_heads=8, num_kv_heads=2, head_dim=128, max_blocks_per_seq=4,
                max_seq_len=64, num_blocks=20, split_blocks=0)
    base.update(kw)
    return L.Shape(**base)


def test_param_count_matches_paper(L):
    assert L.gate_param_count(L.HEAD_PAPER, 2048, 1024) == 28_325_889       # App. A.2
    assert L.gate_param_count(L.HEAD_MLP, 4096, 256) == 4096 * 256 + 2 * 256 + 1


@pytest.mark.parametrize("kw,status", [
    (dict(num_layers=0), -2), (dict(batch=0), -2), (dict(num_q_heads=7), -2), (dict(head_dim=96), -3),
    (dict(num_q_heads=2 * 17, num_kv_heads=2), -3), (dict(block_size=32), -3), (dict(max_seq_len=0), -2),
    (dict(max_blocks_per_seq=3), -2), (dict(num_blocks=0), -2), (dict(split_blocks=3), -2),
    (dict(split_blocks=-2), -2), (dict(layer_stride_kv=20 * 2 * 16 * 128 - 8), -2),
    (dict(layer_stride_kv=20 * 2 * 16 * 128 + 4), -2)])
def test_bad_shapes(L, kw, status):
    with pytest.raises(L.OdaError) as e:
        L.attn_workspace_size(_shape(L, **kw), 4, 16)
    assert e.value.status == status
    assert L.last_error()


def test_workspace_size_scales_with_window(L):
    s = _shape(L, max_seq_len=64 * 1024, max_blocks_per_seq=4096, split_blocks=16)
    small = L.attn_workspace_size(s, 4, 1024)
    full = L.attn_workspace_size(s, 0, 0)
    assert 0 < small <= full and small % 256 == 0 and full % 256 == 0
    # the automatic plan needs no workspace when one workgroup per (layer, request, head) fills the GPU
    big = _shape(L, num_layers=32, batch=1, num_q_heads=32, num_kv_heads=8, max_seq_len=32768,
                 max_blocks_per_seq=2048)
    assert L.attn_workspace_size(big, 0, 0) == 0


def _inputs(L, **kw):
    base = dict(q=0x1000, k_cache=0x2000, v_cache=0x3000, block_table=0x4000, seq_lens=0x5000, scale=0.125)
    base.update(kw)
    return L.inputs(base["q"], base["k_cache"], base["v_cache"], base["block_table"], base["seq_lens"],
                    base["scale"], base.get("k_cur"), base.get("v_cur"))


def _plan_bytes(units, splits, G, D):
    """Workspace of a plan with `splits` splits per unit: ticket words, partial
    outputs and (max, sum) pairs, each rounded up to 256 bytes."""
    up = lambda x: -(-x // 256) * 256
    return 0 if splits <= 1 else up(units * 4) + up(units * splits * G * D * 4) + up(units * splits * G * 2 * 4)


@pytest.mark.parametrize("L_,B,Hq,Hkv,D,n,s,w,splits", [
    (1, 1, 32, 8, 128, 32768, 4, 1024, 7),      # one-layer Local, Llama shape: 66 blocks in splits of 10
    (1, 1, 16, 8, 128, 131072, 4, 2048, 13),    # one-layer Local, decoder shape: 130 blocks in splits of 10
    (1, 1, 16, 8, 128, 4140, 0, 0, 15),         # one-layer Full over 4,140 positions: at most 16 splits
    (1, 1, 32, 8, 128, 32768, 0, 0, 32),        # one-layer Full over 32,768: 32 splits of 64 blocks
    (32, 1, 32, 8, 128, 32768, 4, 1024, 1),     # the stacked call: one split per unit, no workspace
])
def test_automatic_split_plan(L, L_, B, Hq, Hkv, D, n, s, w, splits):
    """The automatic plan (visible through the workspace it asks for): splits
    of at least eight blocks for small calls, more than 16 only while each
    keeps 64 blocks, one split per unit once the units fill the chip."""
    shape = L.Shape(L_, B, Hq, Hkv, D, -(-n // 16), n, 1000, 0)
    assert L.attn_workspace_size(shape, s, w) == _plan_bytes(L_ * B * Hkv, splits, Hq // Hkv, D)


def test_local_rejects_bad_arguments_without_launching(L):
    s = _shape(L, split_blocks=2)           # several splits per request: a workspace is required
    ws_bytes = L.attn_workspace_size(s, 4, 16)
    assert ws_bytes > 0
    cases = [
        (dict(q=None), 0x9000, 0x100000, ws_bytes, 4, 16, -1),
        (dict(k_cur=0x6000), 0x9000, 0x100000, ws_bytes, 4, 16, -1),            # v_cur missing
        (dict(q=0x1008), 0x9000, 0x100000, ws_bytes, 4, 16, -2),                # misaligned
        (dict(scale=0.0), 0x9000, 0x100000, ws_bytes, 4, 16, -2),
        (dict(scale=math.inf), 0x9000, 0x100000, ws_bytes, 4, 16, -2),
        (dict(), None, 0x100000, ws_bytes, 4, 16, -1),                          # out NULL
        (dict(), 0x9000, None, ws_bytes, 4, 16, -4),                            # no workspace
        (dict(), 0x9000, 0x100000, ws_bytes - 1, 4, 16, -4),                    # too small
        (dict(), 0x9000, 0x100010, ws_bytes, 4, 16, -4),                        # misaligned workspace
        (dict(), 0x9000, 0x100000, ws_bytes, -1, 16, -2),
        (dict(), 0x9000, 0x100000, ws_bytes, 4, 0, -2),                         # Local needs a window
    ]
    for kw, out, ws, wb, s_, w_, status in cases:
        with pytest.raises(L.OdaError) as e:
            L.local_decode_attn(s, _inputs(L, **kw), s_, w_, out, None, ws, workspace_bytes=wb, stream=0)
        assert e.value.status == status, (kw, e.value)


def test_full_rejects_bad_arguments(L):
    s = _shape(L, split_blocks=2)
    wb = L.attn_workspace_size(s, 0, 0)
    with pytest.raises(L.OdaError) as e:
        L.full_decode_attn(s, _inputs(L), 0, None, 0x7000, None, 0x9000, None, 0x100000, wb, stream=0)
    assert e.value.status == -1                                            # work_list without n_work
    with pytest.raises(L.OdaError) as e:
        L.full_decode_attn(s, _inputs(L), -5, None, None, None, 0x9000, None, 0x100000, wb, stream=0)
    assert e.value.status == -2


def test_fused_prep_calls_reject_bad_arguments(L):
    """oda_*_decode_attn_qkv: one layer, q / k_cur / v_cur NULL, prep complete and sane."""
    s1 = _shape(L, num_layers=1)
    wb = L.attn_workspace_size(s1, 4, 16)

    def prep(**kw):
        base = dict(qkv=0x3000, q_gain=0x4000, k_gain=0x5000, rms_eps=1e-6, rope_theta=1e6, k_out=0x6000,
                    v_out=0x7000)
        base.update(kw)
        return L.qkv_prep(**base)

    cases = [
        (s1, dict(q=None), prep(qkv=None), -1),                     # qkv missing
        (s1, dict(q=None), prep(v_out=None), -1),                   # k_out without v_out
        (s1, dict(), prep(), -2),                                   # q must be NULL
        (s1, dict(q=None, k_cur=0x6000, v_cur=0x8000), prep(), -2),  # the candidate comes from prep
        (_shape(L, num_layers=2), dict(q=None), prep(), -2),        # one layer only
        (s1, dict(q=None), prep(rope_theta=1.0), -2),
        (s1, dict(q=None), prep(rope_theta=math.nan), -2),
        (s1, dict(q=None), prep(rms_eps=-1e-6), -2),
    ]
    for shape, kw, pr, status in cases:
        wbs = L.attn_workspace_size(shape, 4, 16)
        for call in (L.prepare_local_qkv(shape, _inputs(L, **kw), pr, 4, 16, 0x9000, None, 0x100000, wbs, stream=0),
                     L.prepare_full_qkv(shape, _inputs(L, **kw), pr, 0, None, None, None, 0x9000, None, 0x100000,
                                        L.attn_workspace_size(shape, 0, 0), stream=0)):
            with pytest.raises(L.OdaError) as e:
                call()
            assert e.value.status == status, (kw, e.value)
    # a NULL prep struct
    cs = s1.c()
    inp = _inputs(L, q=None)
    assert L._lib.oda_local_decode_attn_qkv(ctypes.byref(cs), ctypes.byref(inp), None, 4, 16, 0x9000, None,
                                            0x100000, wb, None) == -1


def test_gate_rejects_bad_arguments(L):
    g = L.gate_desc(L.HEAD_PAPER, 64, 16, 0x8000)
    wb = L.gate_workspace_size(g, 4)
    ok = dict(h_prev=0x1000, emb=0x2000, h_local=0x3000, score=0x4000, flags=0x5000)

    def call(gate=g, batch=4, tau=0.0, ws=0x100000, wbytes=wb, **kw):
        a = dict(ok)
        a.update(kw)
        L.recall_gate(gate, batch, a["h_prev"], a["emb"], a["h_local"], tau, None, a["score"], a["flags"],
                      a.get("work_list"), a.get("n_work"), None, ws, wbytes, stream=0)

    for kw, status in [(dict(emb=None), -1), (dict(score=None), -1), (dict(batch=0), -2), (dict(tau=math.nan), -2),
                       (dict(ws=None), -4), (dict(wbytes=wb - 1), -4), (dict(work_list=0x6000), -1),
                       (dict(gate=L.gate_desc(7, 64, 16, 0x8000)), -3), (dict(gate=L.gate_desc(0, 62, 16, 0x8000)), -2),
                       (dict(gate=L.gate_desc(0, 64, 16, 0x8004)), -2)]:
        with pytest.raises(L.OdaError) as e:
            call(**kw)
        assert e.value.status == status, (kw, e.value)
    # the MLP stand-in needs only h_local
    gm = L.gate_desc(L.HEAD_MLP, 64, 16, 0x8000)
    with pytest.raises(L.OdaError) as e:
        L.recall_gate(gm, 4, None, None, None, 0.0, None, 0x4000, 0x5000, None, None, None, 0x100000,
                      L.gate_workspace_size(gm, 4), stream=0)
    assert e.value.status == -1


def test_status_strings(L):
    for s in (0, -1, -2, -3, -4, -5):
        assert L.status_string(s).startswith("ODA_")


def test_commit_rejects_bad_arguments(L):
    s = _shape(L)
    args = dict(k_cache=0x1000, v_cache=0x2000, table=0x3000, seq=0x4000, kl=0x5000, vl=0x6000)

    def call(kw, shape=s):
        a = dict(args)
        a.update(kw)
        L.commit_kv(shape, a["k_cache"], a["v_cache"], a["table"], a["seq"], a["kl"], a["vl"], a.get("kf"),
                    a.get("vf"), None, a.get("advance", True), a.get("ws", 0x8000), a.get("wb", 256), stream=0)

    assert L.commit_workspace_size(s) == 256
    assert L.commit_workspace_size(_shape(L, batch=65)) == 512
    for kw, status in [(dict(k_cache=None), -1), (dict(kl=None), -1), (dict(kf=0x7000), -1),
                       (dict(kl=0x5008), -2), (dict(ws=None), -4), (dict(wb=255), -4), (dict(ws=0x8010), -4)]:
        with pytest.raises(L.OdaError) as e:
            call(kw)
        assert e.value.status == status, (kw, e.value)
    with pytest.raises(L.OdaError) as e:
        call({}, shape=_shape(L, head_dim=96))
    assert e.value.status == -3


def test_ring_elements(L):
    """Direct-ring Local rings: SB = ceil(s/16) sink blocks plus RB = ceil(w/16) + 2
    ring blocks per (layer, request, KV head), each block 16 * D elements."""
    s = _shape(L)                                   # L=2, B=3, Hkv=2, D=128
    per_block = 2 * 3 * 2 * 16 * 128
    assert L.ring_elements(s, 4, 40) == (1 + 5) * per_block
    assert L.ring_elements(s, 0, 16) == (0 + 3) * per_block
    assert L.ring_elements(s, 20, 2048) == (2 + 130) * per_block
    assert L.ring_elements(s, 16, 17) == (1 + 4) * per_block
    for n_sink, window in [(-1, 16), (0, 0)]:
        with pytest.raises(L.OdaError) as e:
            L.ring_elements(s, n_sink, window)
        assert e.value.status == -2


def test_ring_calls_reject_bad_arguments(L):
    s = _shape(L)
    inp = L.inputs(0x1000, None, None, None, 0x4000, 0.1)

    def status_of(fn):
        with pytest.raises(L.OdaError) as e:
            fn()
        return e.value.status

    fill = dict(kc=0x1000, vc=0x2000, t=0x3000, seq=0x4000, kr=0x5000, vr=0x6000, s=4, w=40)

    def do_fill(**kw):
        a = dict(fill)
        a.update(kw)
        L.ring_fill(a.get("shape", s), a["kc"], a["vc"], a["t"], a["seq"], a["s"], a["w"], a["kr"], a["vr"], stream=0)

    for kw, st in [(dict(kc=None), -1), (dict(t=None), -1), (dict(kr=None), -1), (dict(vr=0x6008), -2),
                   (dict(w=0), -2), (dict(s=-1), -2), (dict(shape=_shape(L, head_dim=96)), -3)]:
        assert status_of(lambda: do_fill(**kw)) == st, kw

    def local(inp=inp, kr=0x5000, vr=0x6000, n_sink=4, window=40, out=0x7000, shape=s):
        L.local_decode_attn_ring(shape, inp, kr, vr, n_sink, window, out, None, None, 0, stream=0)

    assert status_of(lambda: local(kr=None)) == -1
    assert status_of(lambda: local(inp=L.inputs(None, None, None, None, 0x4000, 0.1))) == -1
    assert status_of(lambda: local(inp=L.inputs(0x1000, None, None, None, 0x4000, 0.1, 0x8000, None))) == -1
    assert status_of(lambda: local(out=None)) == -1
    assert status_of(lambda: local(vr=0x6004)) == -2
    assert status_of(lambda: local(inp=L.inputs(0x1000, None, None, None, 0x4000, 0.0))) == -2
    assert status_of(lambda: local(window=0)) == -2
    assert status_of(lambda: local(n_sink=-1)) == -2
    assert status_of(lambda: local(shape=_shape(L, num_q_heads=7))) == -2

    def commit(kr=0x5000, vr=0x6000, n_sink=4, window=40, kc=0x1000):
        L.commit_kv_ring(s, kc, 0x2000, 0x3000, 0x4000, 0x9000, 0xa000, None, None, None, True, 0x8000,
                         kr, vr, n_sink, window, workspace_bytes=256, stream=0)

    assert status_of(lambda: commit(kr=None)) == -1
    assert status_of(lambda: commit(vr=0x6002)) == -2
    assert status_of(lambda: commit(window=0)) == -2
    assert status_of(lambda: commit(kc=None)) == -1


def test_decoder_entry_points_reject_bad_arguments(L):
    def status_of(fn):
        with pytest.raises(L.OdaError) as e:
            fn()
        return e.value.status

    w, x, y = 0x10000, 0x20000, 0x30000
    ok = dict(in_features=64, out_features=8, mode=L.DENSE_PLAIN, weight=w, norm_gain=None)

    def dense(batch=2, x_=x, res=None, wl=None, nw=None, **kw):
        a = dict(ok)
        a.update(kw)
        d = L.dense_desc(a["in_features"], a["out_features"], a["mode"], a["weight"], a["norm_gain"])
        return lambda: L.dense_bf16(d, batch, x_, res, y, wl, nw, stream=0)

    assert status_of(dense(weight=None)) == -1
    assert status_of(dense(x_=None)) == -1
    assert status_of(dense(wl=0x40000)) == -1                 # list without its count
    assert status_of(dense(in_features=60)) == -2             # K not a multiple of 8
    assert status_of(dense(batch=0)) == -2
    assert status_of(dense(mode=7)) == -3
    assert status_of(dense(mode=L.DENSE_SWIGLU, res=x)) == -3
    assert status_of(dense(x_=x + 4)) == -2                   # misaligned input
    rope = lambda **kw: (lambda: L.qk_norm_rope(**{**dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                                              qkv=x, q_gain=None, k_gain=None, rms_eps=1e-6,
                                                              rope_theta=1e6, seq_lens=0x50000, q_out=y,
                                                              k_out=0x60000, v_out=0x70000, stream=0), **kw}))
    assert status_of(rope(qkv=None)) == -1
    assert status_of(rope(num_q_heads=7)) == -2
    assert status_of(rope(head_dim=256)) == -3
    assert status_of(rope(rope_theta=1.0)) == -2
    assert status_of(lambda: L.embed_bf16(w, 100, 60, 2, 0x50000, x, stream=0)) == -2
    assert status_of(lambda: L.embed_bf16(None, 100, 64, 2, 0x50000, x, stream=0)) == -1
    assert status_of(lambda: L.copy_rows(2, 6, x, y, stream=0)) == -2
    assert status_of(lambda: L.copy_rows(2, 8, x, y, 0x40000, None, stream=0)) == -1
    g = 0x80000
    assert status_of(lambda: L.rms_norm_rows(2, 8, None, g, 1e-6, y, stream=0)) == -1
    assert status_of(lambda: L.rms_norm_rows(2, 8, x, None, 1e-6, y, stream=0)) == -1
    assert status_of(lambda: L.rms_norm_rows(2, 6, x, g, 1e-6, y, stream=0)) == -2
    assert status_of(lambda: L.rms_norm_rows(2, 8, x, g, -1.0, y, stream=0)) == -2
    assert status_of(lambda: L.rms_norm_rows(2, 8, x + 4, g, 1e-6, y, stream=0)) == -2
    assert status_of(lambda: L.rms_norm_rows(2, 8, x, g, 1e-6, y, 0x40000, None, stream=0)) == -1
    assert status_of(lambda: L.argmax(2, 10, x, y, stream=0)) == -2
    assert status_of(lambda: L.argmax(0, 8, x, y, stream=0)) == -2


def test_stream_read_rejects_bad_arguments(L):
    def status_of_read(src=0x10000, nbytes=4096, sink=0x20000, groups=0):
        with pytest.raises(L.OdaError) as e:
            L.stream_read(src, nbytes, sink, groups, stream=0)
        return e.value.status

    assert status_of_read(src=None) == -1
    assert status_of_read(sink=None) == -1
    assert status_of_read(src=0x10008) == -2                  # misaligned
    assert status_of_read(nbytes=4100) == -2                  # not a multiple of 16
    assert status_of_read(groups=-1) == -2
    L.stream_read(0x10000, 0, 0x20000, 0, stream=0)           # nothing to read: no launch


def test_library_shares_torchs_hip_runtime():
    """Importing the binding before anything else still leaves one HIP
    runtime in the process (torch's): a second one would find no GPU."""
    code = ("import paper_2609_20734_amd._lib, torch\n"
            "maps = open('/proc/self/maps').read()\n"
            "libs = {l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}\n"
            "print(len(libs), sorted(libs))\n")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.startswith("1 "), r.stdout
