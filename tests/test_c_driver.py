"""A decode step driven from C: tests/c_abi/decode_step.c includes
include/oda.h, links liboda.so and calls Local attention, the recall gate
(MLP stand-in) and Full attention over the compacted list.  The inputs come
from the seeded generators; the outputs are checked against the fp64 oracle."""
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

import oda_synth as S
from harness import FLAG_BORDER, LSE_ABS, check_close, note_flags
from oracle import attention as OA
from oracle import gate as OG

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_20734_amd")


def _compile(exe):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    cmd = [cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "c_abi", "decode_step.c"),
           "-L", PKG, "-loda", "-L", "/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath," + PKG, "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr


def test_decode_step_from_c(tmp_path):
    if not os.path.exists(os.path.join(PKG, "liboda.so")):
        pytest.fail("liboda.so is not built")
    exe = str(tmp_path / "decode_step")
    _compile(exe)

    seed = 77
    L, B, Hq, Hkv, D = 2, 5, 8, 2, 64
    n_sink, window = 4, 96
    seq = np.array([1500, 97, 1, 640, 333], dtype=np.int32)
    d, h = 128, 32
    mb = int(np.ceil(seq.max() / 16))
    q = S.normal_bf16(S.rng(seed, S.STREAM_Q), (L, B, Hq, D))
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq, mb, permute=True, extra_blocks=3)
    k, v = S.kv_cache(seed, L, nb, Hkv, D)
    params = S.gate_params(seed, "mlp", d, h).astype(np.float32)
    _, _, hl = (x[0] for x in S.gate_inputs(seed, 1, B, d))
    hl = hl.astype(np.float32)
    score_ref = OG.mlp_score(params.astype(np.float64), d, h, hl.astype(np.float64))
    tau = float(np.median(score_ref))       # about half the requests take Full
    scale = 1.0 / np.sqrt(D)

    inp = tmp_path / "inputs.bin"
    with open(inp, "wb") as f:
        f.write(np.array([L, B, Hq, Hkv, D, mb, int(seq.max()), nb, n_sink, window, d, h], np.int32).tobytes())
        f.write(np.array([tau, scale, 1e-6], np.float32).tobytes())
        for a, dt in ((q, np.uint16), (k, np.uint16), (v, np.uint16), (table, np.int32), (seq, np.int32),
                      (params, np.float32), (hl, np.float32)):
            assert a.dtype == dt
            f.write(np.ascontiguousarray(a).tobytes())
    outp = tmp_path / "outputs.bin"
    print(f"running the C driver: L={L} B={B} seq={seq.tolist()}", flush=True)
    res = subprocess.run([exe, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr

    raw = open(outp, "rb").read()
    off = 0

    def take(count, dtype):
        nonlocal off
        a = np.frombuffer(raw, dtype=dtype, count=count, offset=off)
        off += a.nbytes
        return a

    out = take(L * B * Hq * D, np.float32).reshape(L, B, Hq, D)
    lse = take(L * B * Hq, np.float32).reshape(L, B, Hq)
    score = take(B, np.float32)
    flags = take(B, np.int32)
    work = take(B, np.int32)
    n_work = int(take(1, np.int32)[0])
    assert off == len(raw)

    scale_ = max(1.0, float(np.abs(score_ref).max()))
    assert np.max(np.abs(score - score_ref)) <= 1e-4 * scale_
    want = OG.decide(score_ref, tau)
    border = np.abs(score_ref - tau) < FLAG_BORDER
    note_flags("C driver", border, flags.astype(bool) != want)
    assert not ((flags.astype(bool) != want) & ~border).any()
    assert n_work == int(flags.sum()) and np.array_equal(work[:n_work], np.flatnonzero(flags))

    local, local_lse, _ = OA.decode_attention(q, k, v, table, seq, lambda n: OA.local_set(n, n_sink, window), scale)
    full, full_lse, _ = OA.decode_attention(q, k, v, table, seq, OA.full_set, scale)
    for b in range(B):
        ref, ref_lse = (full, full_lse) if flags[b] else (local, local_lse)
        check_close(out[:, b], ref[:, b], what=f"request {b} ({'Full' if flags[b] else 'Local'})")
        assert np.max(np.abs(lse[:, b] - ref_lse[:, b])) <= LSE_ABS
