"""Shared plumbing for the GPU tests: seeded inputs on the host (oda_synth),
copies on the device, calls through the C ABI (paper_2609_20734_amd), and the
tolerance checks.  Expected values always come from the fp64 oracle.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oda_synth as S
from oracle import attention as OA

# Bars: the attention output must match the fp64 oracle within max-abs 2e-3 and
# relative-L2 1e-3; internally we hold the kernels to 1e-4 max-abs (bf16 inputs
# are exact, accumulation is fp32, so the expected error is ~1e-6).
MAX_ABS = 2e-3
REL_L2 = 1e-3
MAX_ABS_INTERNAL = 1e-4
LSE_ABS = 1e-4
FLAG_BORDER = 1e-4


# Flag decisions whose fp64 score lies within FLAG_BORDER of the threshold are
# exempt from the bit-exact comparison (the kernel decides in fp32); they are
# counted here and reported at the end of the session (conftest).
FLAG_TALLY = {"decisions": 0, "borderline": 0, "mismatched_borderline": 0, "where": {}}


def note_flags(where: str, border, mismatch=None) -> int:
    """Count one comparison's flag decisions: `border` marks the decisions
    within FLAG_BORDER of the threshold, `mismatch` (optional) those where
    the kernel and the oracle disagree.  Returns the borderline count."""
    border = np.asarray(border, dtype=bool)
    nb = int(border.sum())
    FLAG_TALLY["decisions"] += int(border.size)
    FLAG_TALLY["borderline"] += nb
    if mismatch is not None:
        FLAG_TALLY["mismatched_borderline"] += int((np.asarray(mismatch, dtype=bool) & border).sum())
    if nb:
        FLAG_TALLY["where"][where] = FLAG_TALLY["where"].get(where, 0) + nb
        print(f"[flags] {where}: {nb} borderline decision(s) of {border.size}", flush=True)
    return nb


def need_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("this test needs an MI355X")
    import paper_2609_20734_amd as P
    return P


def dev_u16(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def dev_f32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).cuda()


def check_close(got, ref, what="out", internal=True):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: nonfinite values"
    err = np.abs(got - ref)
    max_abs = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    assert max_abs <= MAX_ABS, f"{what}: max-abs {max_abs:.3e} > {MAX_ABS}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3e} > {REL_L2}"
    if internal:
        assert max_abs <= MAX_ABS_INTERNAL, f"{what}: max-abs {max_abs:.3e} above the internal bar {MAX_ABS_INTERNAL}"
    return max_abs, rel


class AttnProblem:
    """A paged decode-attention problem: host copies for the oracle, device
    copies for the kernels (identical bits)."""

    def __init__(self, seed, L, B, Hq, Hkv, D, seq, permute=True, cur=False, split_blocks=0,
                 extra_blocks=5, max_blocks_per_seq=None, max_len=None):
        self.P = need_gpu()
        self.L, self.B, self.Hq, self.Hkv, self.D = L, B, Hq, Hkv, D
        self.seq = np.asarray(seq, dtype=np.int32)
        self.q = S.normal_bf16(S.rng(seed, S.STREAM_Q), (L, B, Hq, D))
        max_len = max_len or int(self.seq.max())
        mb = max_blocks_per_seq or max(1, int(math.ceil(max_len / 16)))
        self.table, self.nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), self.seq, mb, permute=permute,
                                                  extra_blocks=extra_blocks)
        self.k, self.v = S.kv_cache(seed, L, self.nb, Hkv, D)
        self.kc = self.vc = None
        if cur:
            self.kc = S.normal_bf16(S.rng(seed, S.STREAM_KCUR), (L, B, Hkv, D))
            self.vc = S.normal_bf16(S.rng(seed, S.STREAM_VCUR), (L, B, Hkv, D))
        self.scale = 1.0 / math.sqrt(D)
        self.shape = self.P.Shape(L, B, Hq, Hkv, D, mb, max_len, self.nb, split_blocks)
        self.upload()

    def upload(self):
        self.dq, self.dk, self.dv = dev_u16(self.q), dev_u16(self.k), dev_u16(self.v)
        self.dtable, self.dseq = dev_i32(self.table), dev_i32(self.seq)
        self.dkc = dev_u16(self.kc) if self.kc is not None else None
        self.dvc = dev_u16(self.vc) if self.vc is not None else None
        self.inp = self.P.inputs(self.dq, self.dk, self.dv, self.dtable, self.dseq, self.scale, self.dkc, self.dvc)

    def new_out(self, fill=0.0):
        out = torch.full((self.L, self.B, self.Hq, self.D), fill, dtype=torch.float32, device="cuda")
        lse = torch.full((self.L, self.B, self.Hq), fill, dtype=torch.float32, device="cuda")
        return out, lse

    def run_local(self, n_sink, window, out=None, lse=None):
        if out is None:
            out, lse = self.new_out(np.nan)
        ws = torch.zeros(self.P.attn_workspace_size(self.shape, n_sink, window), dtype=torch.uint8, device="cuda")
        self.P.local_decode_attn(self.shape, self.inp, n_sink, window, out, lse, ws)
        torch.cuda.synchronize()
        return out, lse

    def run_full(self, native_window=0, flags=None, work_list=None, n_work=None, out=None, lse=None):
        if out is None:
            out, lse = self.new_out(np.nan)
        ws = torch.zeros(self.P.attn_workspace_size(self.shape, 0, native_window), dtype=torch.uint8,
                         device="cuda")
        self.P.full_decode_attn(self.shape, self.inp, native_window, flags, work_list, n_work, out, lse, ws)
        torch.cuda.synchronize()
        return out, lse

    def oracle(self, positions_of, requests=None):
        return OA.decode_attention(self.q, self.k, self.v, self.table, self.seq, positions_of, self.scale,
                                   k_cur=self.kc, v_cur=self.vc, requests=requests)

    def oracle_local(self, n_sink, window, requests=None):
        return self.oracle(lambda n: OA.local_set(n, n_sink, window), requests)

    def oracle_full(self, native_window=0, requests=None):
        return self.oracle(lambda n: OA.native_window_set(n, native_window), requests)
