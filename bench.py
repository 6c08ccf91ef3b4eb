#!/usr/bin/env python3
"""Benchmark of the ODA decode-step hot path on one MI355X.

A step is one pass of the whole path over one batch: Local decode attention
for every layer and request, the recall gate (score + device predicate +
compaction), and Full decode attention for the flagged requests only, all on
one stream.  The recall rate rho is swept by the threshold tau (calibrated on
the gate's scores over the K timed steps) or, for the mixed-length batch, by
Bernoulli schedules of forced flags (threshold-driven rates reported beside
them), and compared against the always-Full baseline (Full for every request,
no Local, no gate).

Timing: every step is bracketed by HIP events on the stream the library
launches on.  Headline ("cold") numbers read a 1 GiB scratch buffer between
steps, outside the events, so the 256 MB Infinity Cache holds no KV or gate
weights at the start of a step; each operating point runs `reps` repetitions
of K steps and reports the median of the repetitions' means (with their min
and max); "warm" numbers run the K steps back to back.  Two launch modes:
stacked (one call covers every layer of a group; the metric) and per-layer
(one call per layer, eager and as a captured HIP graph; the realism check).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--reps R] [--config mixed] [--head paper|mlp]

Prints one JSON line: the headline value (µs per step at the recall rate
nearest 0.1), the per-rate sweep for both recall heads, the per-layer launch
mode, the decode loop, Local with and without sinks, the streaming-read
ceiling, the roofline of the dominant kernel and the CPU oracle baseline (one
thread and a process pool, timed before the GPU is touched).

    python bench.py --decoder [--lengths 4139,15918,...]

instead times whole decode steps of a synthetic Qwen3-1.7B-shaped decoder
(App. A.6's cost model: backbone, attention, recall head, output) at batch
one: native Full, standalone Local and ODA with the first 2, 4 or 8 of every
16 steps prescribed Full, as tokens/s, and prints one JSON line of those.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn µs/step + achieved HBM GB/s vs always-Full, recall rate 0-100%"
HBM_PEAK_GBS = 8000.0
HEADLINE_RHO = 0.1
FLAG_BORDER = 1e-4      # |score - tau| below this: a borderline decision (fp32 kernel vs fp64 oracle)
ROOFLINE_REPS = 20
ROOFLINE_KERNEL = "attn_split_kernel<128, false>"
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_20734_amd", "csrc", "attention.hip")


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"full_split_{workload}_traffic.txt")


def source_sha256() -> str:
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload: str, bytes_per_launch: int):
    """HBM bytes per launch of the roofline kernel from the committed PMC summary
    of this workload, or None if there is none, if it was taken on another
    launch size, or if the kernel source changed since it was taken."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha256() or vals.get("workload_name") != workload:
        return None
    try:
        if int(vals["algorithmic_bytes_per_launch"]) != int(bytes_per_launch):
            return None
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class StackState:
    """Device buffers of one layer group (shared block table)."""

    def __init__(self, P, wl, stack, seq, table, num_blocks, mb, max_len, seed, dev, split_blocks):
        import torch

        import oda_synth as S
        self.stack = stack
        L, B, Hq, Hkv, D = stack.num_layers, wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        self.shape = P.Shape(L, B, Hq, Hkv, D, mb, max_len, num_blocks, split_blocks)
        self.k = torch.empty((L, num_blocks, Hkv, D // 8, 16, 8), dtype=torch.bfloat16, device=dev)
        self.v = torch.empty((L, num_blocks, Hkv, D, 16), dtype=torch.bfloat16, device=dev)
        S.fill_normal_bf16_(self.k, seed, S.STREAM_K + 100 * len(stack.name))
        S.fill_normal_bf16_(self.v, seed, S.STREAM_V + 100 * len(stack.name))
        q = S.normal_bf16(S.rng(seed + len(stack.name), S.STREAM_Q), (L, B, Hq, D))
        self.q = torch.from_numpy(q.view(np.int16)).to(dev)
        self.table = table
        self.seq = seq
        self.inp = P.inputs(self.q, self.k, self.v, table, seq, 1.0 / math.sqrt(D))
        self.out = torch.zeros((L, B, Hq, D), dtype=torch.float32, device=dev)
        self.lse = torch.zeros((L, B, Hq), dtype=torch.float32, device=dev)
        loc_w = stack.native_window if not stack.gated else stack.local_window
        loc_s = 0 if not stack.gated else stack.local_sink
        self.local_args = (loc_s, loc_w)
        self.ws_local = torch.zeros(P.attn_workspace_size(self.shape, loc_s, loc_w), dtype=torch.uint8, device=dev)
        self.ws_full = torch.zeros(P.attn_workspace_size(self.shape, 0, stack.native_window), dtype=torch.uint8,
                                   device=dev)
        self.k_ring = self.v_ring = None

    def make_rings(self, P, dev):
        """Direct-ring Local workspace of this layer group (filled by Bench.fill_rings)."""
        import torch
        n = P.ring_elements(self.shape, *self.local_args)
        self.k_ring = torch.empty(n, dtype=torch.int16, device=dev)
        self.v_ring = torch.empty(n, dtype=torch.int16, device=dev)


class Bench:
    def __init__(self, wl, head, seed, steps, split_blocks=0, growth=0, local="ring"):
        import torch

        import oda_synth as S
        import paper_2609_20734_amd as P
        self.P, self.torch, self.wl, self.seed, self.K = P, torch, wl, seed, steps
        dev = torch.device("cuda:0")
        self.dev = dev
        B = wl.batch
        seq = workload_seq_lens(wl, seed)
        self.seq_host = seq
        self.growth = growth     # positions a decode loop may append (blocks reserved in the table)
        mb = int(math.ceil((seq.max() + growth) / 16))
        table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq + growth, mb, permute=wl.permute)
        need = sum(st.num_layers for st in wl.stacks) * nb * wl.num_kv_heads * wl.head_dim * 16 * 2 * 2
        free, total = torch.cuda.mem_get_info()
        log(f"[bench] {wl.name}: KV {need / 1e9:.2f} GB, device free {free / 1e9:.1f} GB")
        if need > free - 8e9:
            raise SystemExit(f"workload needs {need / 1e9:.1f} GB of KV, only {free / 1e9:.1f} GB free")
        self.dtable = torch.from_numpy(table).to(dev)
        self.dseq = torch.from_numpy(seq).to(dev)
        self.stacks = [StackState(P, wl, st, self.dseq, self.dtable, nb, mb, int(seq.max()) + growth, seed, dev,
                                  split_blocks) for st in wl.stacks]
        # Local reads the direct-ring workspace (App. A.5), or the paged cache
        self.local = local
        if local == "ring":
            for st in self.stacks:
                st.make_rings(P, dev)
            self.fill_rings()
        # gate
        h, e, l = S.gate_inputs(seed, steps, B, wl.d_model)
        self.h = torch.from_numpy(h).to(dev)
        self.e = torch.from_numpy(e).to(dev)
        self.l = torch.from_numpy(l).to(dev)
        self.set_head(head)
        self.score = torch.zeros(B, dtype=torch.float32, device=dev)
        self.flags = torch.zeros(B, dtype=torch.int32, device=dev)
        self.work = torch.zeros(B, dtype=torch.int32, device=dev)
        self.n_work = torch.zeros(1, dtype=torch.int32, device=dev)
        self.counter = torch.zeros(1, dtype=torch.int64, device=dev)
        # staging copies of one step's gate inputs and forced flags (per-layer launch mode)
        self.h_stage = torch.zeros((B, wl.d_model), dtype=torch.float32, device=dev)
        self.e_stage = torch.zeros_like(self.h_stage)
        self.l_stage = torch.zeros_like(self.h_stage)
        self.f_stage = torch.zeros(B, dtype=torch.int32, device=dev)
        self.sink = torch.zeros(64, dtype=torch.int32, device=dev)
        # 1 GiB read between steps evicts the 256 MB Infinity Cache with clean lines
        # (a write flush would leave dirty lines for the next step to write back)
        self.flush_buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)

    def flush(self):
        self.flush_buf.max()

    def fill_rings(self):
        """(Re)fill every layer group's rings from the paged cache at the current lengths."""
        for st in self.stacks:
            if st.k_ring is not None:
                self.P.ring_fill(st.shape, st.k, st.v, self.dtable, self.dseq, *st.local_args, st.k_ring, st.v_ring)

    def local_call(self, st, layer=None, k_cur=None, v_cur=None, ws=None):
        """The pre-marshalled Local call of a layer group (all its layers, or one
        layer with a one-layer shape), through the rings or the paged cache."""
        P = self.P
        scale = 1.0 / math.sqrt(self.wl.head_dim)
        shape, q, out, lse, kr, vr, k, v = st.shape, st.q, st.out, st.lse, st.k_ring, st.v_ring, st.k, st.v
        if layer is not None:
            s = st.shape
            shape = P.Shape(1, s.batch, s.num_q_heads, s.num_kv_heads, s.head_dim, s.max_blocks_per_seq,
                            s.max_seq_len, s.num_blocks, s.split_blocks)
            q, out, lse, k, v = q[layer], out[layer], lse[layer], k[layer], v[layer]
            if kr is not None:
                kr, vr = kr.view(st.stack.num_layers, -1)[layer], vr.view(st.stack.num_layers, -1)[layer]
        ws = st.ws_local if ws is None else ws
        if self.local == "ring":
            return P.prepare_local_ring(shape, P.inputs(q, None, None, None, self.dseq, scale, k_cur, v_cur), kr, vr,
                                        *st.local_args, out, lse, ws)
        return P.prepare_local(shape, P.inputs(q, k, v, self.dtable, self.dseq, scale, k_cur, v_cur),
                               *st.local_args, out, lse, ws)

    def set_head(self, head):
        """Recall head used by the steps: the App. A.2 form ("paper") or the MLP stand-in."""
        import torch

        import oda_synth as S
        P, wl = self.P, self.wl
        self.head = head
        kind = P.HEAD_PAPER if head == "paper" else P.HEAD_MLP
        params = S.gate_params(self.seed, head, wl.d_model, wl.d_hidden)
        self.params = torch.from_numpy(params).to(self.dev)
        self.gate = P.gate_desc(kind, wl.d_model, wl.d_hidden, self.params, 1e-6)
        self.ws_gate = torch.zeros(P.gate_workspace_size(self.gate, wl.batch), dtype=torch.uint8, device=self.dev)

    # -- calls ---------------------------------------------------------------
    def step_calls(self, tau, forced=None, gated_only=False):
        """Per step t: the list of pre-marshalled calls of one decode step.
        gated_only: the Full retry covers only the gated layer groups (natively
        windowed layers keep their Local result, which is already native)."""
        P = self.P
        local = [self.local_call(s) for s in self.stacks]
        full = [P.prepare_full(s.shape, s.inp, s.stack.native_window, None, self.work, self.n_work, s.out, s.lse,
                               s.ws_full) for s in self.stacks if s.stack.gated or not gated_only]
        steps = []
        for t in range(self.K):
            fo = None if forced is None else forced[t]
            g = P.prepare_gate(self.gate, self.wl.batch, self.h[t], self.e[t], self.l[t], tau, fo, self.score,
                               self.flags, self.work, self.n_work, self.counter, self.ws_gate)
            steps.append(local + [g] + full)
        return steps

    def decode_loop(self, firsts=(0, 2, 4, 8, 16), period=16, reps=4):
        """The paper's runtime protocol (App. B.7) as a growing-context loop: a
        device-side schedule selects Full for the first k of every `period`
        steps, the gate still runs every step, and each step commits the
        selected candidate (Local or Full current-position K/V of every layer)
        so the context grows by one.  One period is captured as a HIP graph and
        replayed `reps` times back to back (warm, like the paper's throughput
        measurement); the same period launched eagerly is timed too."""
        import oda_synth as S
        torch, P, wl = self.torch, self.P, self.wl
        B = wl.batch
        assert self.growth >= period * (reps + 2), "table has no room for the loop"
        cands = []
        for si, st in enumerate(self.stacks):
            shp = (period, st.stack.num_layers, B, wl.num_kv_heads, wl.head_dim)
            c = [torch.empty(shp, dtype=torch.bfloat16, device=self.dev) for _ in range(4)]
            for i, x in enumerate(c):
                S.fill_normal_bf16_(x, self.seed + 17 * si + i, S.STREAM_KCUR)
            cands.append(c)
        scale = 1.0 / math.sqrt(wl.head_dim)
        seq0 = self.dseq.clone()
        ws_commit = torch.zeros(P.commit_workspace_size(self.stacks[-1].shape), dtype=torch.uint8, device=self.dev)
        res = []

        def reset():
            # lengths back to the start; rings rebuilt (commits past the start overwrote ring blocks the
            # window at the start still reads), the paged cache below the start is intact
            self.dseq.copy_(seq0)
            self.fill_rings()

        def one_period(forced):
            for t in range(period):
                for st, (kl, vl, kf, vf) in zip(self.stacks, cands):
                    self.local_call(st, k_cur=kl[t], v_cur=vl[t])()
                P.recall_gate(self.gate, B, self.h[t % self.K], self.e[t % self.K], self.l[t % self.K], 0.0,
                              forced[t], self.score, self.flags, self.work, self.n_work, self.counter, self.ws_gate)
                for st, (kl, vl, kf, vf) in zip(self.stacks, cands):
                    inp = P.inputs(st.q, st.k, st.v, self.dtable, self.dseq, scale, kf[t], vf[t])
                    P.full_decode_attn(st.shape, inp, st.stack.native_window, None, self.work, self.n_work,
                                       st.out, st.lse, st.ws_full)
                for i, (st, (kl, vl, kf, vf)) in enumerate(zip(self.stacks, cands)):
                    if st.k_ring is not None:
                        P.commit_kv_ring(st.shape, st.k, st.v, self.dtable, self.dseq, kl[t], vl[t], kf[t], vf[t],
                                         self.flags, i == len(self.stacks) - 1, ws_commit, st.k_ring, st.v_ring,
                                         *st.local_args)
                    else:
                        P.commit_kv(st.shape, st.k, st.v, self.dtable, self.dseq, kl[t], vl[t], kf[t], vf[t],
                                    self.flags, i == len(self.stacks) - 1, ws_commit)

        for k in firsts:
            sched = np.stack([S.periodic_schedule(period, k)] * B, axis=1).astype(np.int32)
            forced = torch.from_numpy(sched).to(self.dev)
            # eager: launched from the host every period
            reset()
            one_period(forced)
            torch.cuda.synchronize()
            reset()
            self.counter.zero_()
            a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                one_period(forced)
            b_.record()
            torch.cuda.synchronize()
            eager_us = a.elapsed_time(b_) * 1e3 / (reps * period)
            recalled = int(self.counter.item())
            # graph: the whole period captured once, replayed
            reset()
            g = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                one_period(forced)
            reset()
            g.replay()
            torch.cuda.synchronize()
            reset()
            torch.cuda.synchronize()
            a.record()
            for _ in range(reps):
                g.replay()
            b_.record()
            torch.cuda.synchronize()
            graph_us = a.elapsed_time(b_) * 1e3 / (reps * period)
            grown = int((self.dseq - seq0).max().item())
            res.append(dict(first_k=k, rho=k / period, recalled=recalled, steps=reps * period, eager_us=eager_us,
                            graph_us=graph_us, context_growth=grown))
            log(f"[bench] decode loop first {k}/{period} Full: eager {eager_us:.1f} us/step, "
                f"graph {graph_us:.1f} us/step, recalled {recalled}/{reps * period * B}")
            del g
        reset()
        return res

    def full_calls(self):
        P = self.P
        full = [P.prepare_full(s.shape, s.inp, s.stack.native_window, None, None, None, s.out, s.lse, s.ws_full)
                for s in self.stacks]
        return [full] * self.K

    def step_flags(self, tau, forced=None):
        """The gate's flags for each of the K steps at one operating point
        (the gate alone, outside any timed region): int32 [K][B]."""
        torch = self.torch
        B = self.wl.batch
        out = torch.zeros((self.K, B), dtype=torch.int32, device=self.dev)
        work = torch.zeros(B, dtype=torch.int32, device=self.dev)
        n_work = torch.zeros(1, dtype=torch.int32, device=self.dev)
        for t in range(self.K):
            self.P.recall_gate(self.gate, B, self.h[t], self.e[t], self.l[t], tau,
                               None if forced is None else forced[t], self.score, out[t], work, n_work, None,
                               self.ws_gate)
        return out.cpu().numpy()

    def scores(self):
        """Gate scores of all K steps (tau = +inf), for threshold calibration."""
        out = np.zeros((self.K, self.wl.batch))
        for t in range(self.K):
            self.P.recall_gate(self.gate, self.wl.batch, self.h[t], self.e[t], self.l[t], math.inf, None,
                               self.score, self.flags, None, None, None, self.ws_gate)
            out[t] = self.score.cpu().numpy()
        return out

    # -- timing --------------------------------------------------------------
    def timed(self, steps, warmup, cold=True, pre=None):
        """Time each of the K call lists in `steps` (one decode step each)
        between HIP events; pre(t), if given, runs before step t's start event
        (after the cache flush)."""
        torch = self.torch
        for t in range(warmup):
            if pre is not None:
                pre(t % len(steps))
            for c in steps[t % len(steps)]:
                c()
        torch.cuda.synchronize()
        self.counter.zero_()
        K = len(steps)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
        wall0 = time.perf_counter()
        t_all0 = torch.cuda.Event(enable_timing=True)
        t_all1 = torch.cuda.Event(enable_timing=True)
        t_all0.record()
        for t in range(K):
            if cold:
                self.flush()
            if pre is not None:
                pre(t)
            evs[t][0].record()
            for c in steps[t]:
                c()
            evs[t][1].record()
        t_all1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        per = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])      # us
        return dict(us_mean=float(per.mean()), us_median=float(np.median(per)), us_min=float(per.min()),
                    us_max=float(per.max()), bracket_us=float(t_all0.elapsed_time(t_all1) * 1e3 / K),
                    wall_us=wall * 1e6 / K, per_step=per, recalled=int(self.counter.item()))

    def local_layout(self, reps=20):
        """Local attention alone (every stack, cold) reading the window through
        the permuted block table, through a contiguous one (identity table,
        same cache, same lengths), and from the direct-ring workspace
        (oda_local_decode_attn_ring over rings filled from the same cache: no
        table at all); then the same for one layer of the first stack, where
        the table lookup is a larger share of a call."""
        import oda_synth as S
        torch, P = self.torch, self.P
        seq = self.seq_host + self.growth
        mb = self.stacks[0].shape.max_blocks_per_seq
        ident, nb = S.paged_block_table(S.rng(self.seed, S.STREAM_TABLE), seq, mb, permute=False)
        assert nb == self.stacks[0].shape.num_blocks
        dident = torch.from_numpy(ident).to(self.dev)
        scale = 1.0 / math.sqrt(self.wl.head_dim)
        res = {}
        for name, table in (("permuted", self.dtable), ("contiguous", dident)):
            calls = [P.prepare_local(st.shape, P.inputs(st.q, st.k, st.v, table, self.dseq, scale), *st.local_args,
                                     st.out, st.lse, st.ws_local) for st in self.stacks]
            res[f"{name}_us"] = self.kernel_time(calls, reps, cold=True)
        rings = []
        for st in self.stacks:
            if st.k_ring is not None:
                rings.append((st.k_ring, st.v_ring))
                continue
            n = P.ring_elements(st.shape, *st.local_args)
            kr = torch.empty(n, dtype=torch.int16, device=self.dev)
            vr = torch.empty(n, dtype=torch.int16, device=self.dev)
            P.ring_fill(st.shape, st.k, st.v, self.dtable, self.dseq, *st.local_args, kr, vr)
            rings.append((kr, vr))
        calls = [P.prepare_local_ring(st.shape, P.inputs(st.q, None, None, None, self.dseq, scale), kr, vr,
                                      *st.local_args, st.out, st.lse, st.ws_local)
                 for st, (kr, vr) in zip(self.stacks, rings)]
        res["ring_us"] = self.kernel_time(calls, reps, cold=True)
        res["ring_bytes"] = int(sum(2 * r[0].numel() * 2 for r in rings))
        # one layer of the first stack (the per-layer launch mode's Local call)
        st, (kr, vr) = self.stacks[0], rings[0]
        sh = st.shape
        one = P.Shape(1, sh.batch, sh.num_q_heads, sh.num_kv_heads, sh.head_dim, sh.max_blocks_per_seq,
                      sh.max_seq_len, sh.num_blocks, sh.split_blocks)
        ws1 = torch.zeros(max(256, P.attn_workspace_size(one, *st.local_args)), dtype=torch.uint8, device=self.dev)
        paged1 = P.prepare_local(one, P.inputs(st.q[0], st.k, st.v, self.dtable, self.dseq, scale), *st.local_args,
                                 st.out[0], st.lse[0], ws1)
        ring1 = P.prepare_local_ring(one, P.inputs(st.q[0], None, None, None, self.dseq, scale), kr, vr,
                                     *st.local_args, st.out[0], st.lse[0], ws1)
        res["one_layer_permuted_us"] = self.kernel_time([paged1], reps, cold=True)
        res["one_layer_ring_us"] = self.kernel_time([ring1], reps, cold=True)
        del rings, calls, kr, vr
        torch.cuda.empty_cache()
        return res

    # -- per-layer launch mode --------------------------------------------------
    def _layer_state(self):
        """One-layer shapes, per-layer inputs and workspaces (built once)."""
        if getattr(self, "_layers", None) is None:
            torch, P = self.torch, self.P
            scale = 1.0 / math.sqrt(self.wl.head_dim)
            self._layers = []
            for st in self.stacks:
                s = st.shape
                sh = P.Shape(1, s.batch, s.num_q_heads, s.num_kv_heads, s.head_dim, s.max_blocks_per_seq,
                             s.max_seq_len, s.num_blocks, s.split_blocks)
                ws_l = torch.zeros(max(256, P.attn_workspace_size(sh, *st.local_args)), dtype=torch.uint8,
                                   device=self.dev)
                ws_f = torch.zeros(max(256, P.attn_workspace_size(sh, 0, st.stack.native_window)),
                                   dtype=torch.uint8, device=self.dev)
                ins = [P.inputs(st.q[l], st.k[l], st.v[l], self.dtable, self.dseq, scale)
                       for l in range(st.stack.num_layers)]
                self._layers.append((st, sh, ws_l, ws_f, ins))
        return self._layers

    def per_layer_calls(self, tau, forced, split=False):
        """One decode step as one call per layer: every layer's Local, the gate
        (reading the staged inputs), every layer's Full over the compacted list
        (split: the Local + gate calls and the Full calls as two lists)."""
        P = self.P
        calls = []
        for st, sh, ws_l, _, ins in self._layer_state():
            calls += [self.local_call(st, layer=l, ws=ws_l) for l in range(len(ins))]
        calls.append(P.prepare_gate(self.gate, self.wl.batch, self.h_stage, self.e_stage, self.l_stage, tau,
                                    self.f_stage if forced is not None else None, self.score, self.flags,
                                    self.work, self.n_work, self.counter, self.ws_gate))
        full = []
        for st, sh, _, ws_f, ins in self._layer_state():
            full += [P.prepare_full(sh, inp, st.stack.native_window, None, self.work, self.n_work, st.out[l],
                                    st.lse[l], ws_f) for l, inp in enumerate(ins)]
        return (calls, full) if split else calls + full

    def per_layer(self, tau, forced, warmup):
        """Per-layer launches of the K steps, eager and replayed as one captured
        HIP graph per step shape (gate inputs staged before each step, outside
        the events), and eager with a host branch: the Full calls are launched
        only if the host, after one synchronisation on the device's count of
        flagged requests, sees any (the branch of Alg. 1).  Returns (eager,
        graph, host-branch) timing dicts."""
        torch = self.torch
        K = self.K

        def pre(t):
            self.h_stage.copy_(self.h[t])
            self.e_stage.copy_(self.e[t])
            self.l_stage.copy_(self.l[t])
            if forced is not None:
                self.f_stage.copy_(forced[t])

        calls = self.per_layer_calls(tau, forced)
        eager = self.timed([calls] * K, warmup, cold=True, pre=pre)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for c in self.per_layer_calls(tau, forced):     # prepared on the capture stream
                c()
        graph = self.timed([[g.replay]] * K, warmup, cold=True, pre=pre)
        del g
        first, full = self.per_layer_calls(tau, forced, split=True)
        n_host = torch.zeros(1, dtype=torch.int32).pin_memory()

        def branch():
            n_host.copy_(self.n_work, non_blocking=True)
            torch.cuda.current_stream().synchronize()
            if int(n_host[0]) > 0:
                for c in full:
                    c()
        branched = self.timed([first + [branch]] * K, warmup, cold=True, pre=pre)
        return eager, graph, branched

    def per_layer_full(self, warmup):
        """Always-Full in the per-layer launch mode: one Full call per layer over
        every request, no Local, no gate; eager and as a captured graph."""
        torch, P = self.torch, self.P

        def calls():
            out = []
            for st, sh, _, ws_f, ins in self._layer_state():
                out += [P.prepare_full(sh, inp, st.stack.native_window, None, None, None, st.out[l], st.lse[l],
                                       ws_f) for l, inp in enumerate(ins)]
            return out

        eager = self.timed([calls()] * self.K, warmup, cold=True)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for c in calls():
                c()
        graph = self.timed([[g.replay]] * self.K, warmup, cold=True)
        del g
        return eager, graph

    # -- single measurements -------------------------------------------------------
    def local_sinks(self, reps=20):
        """Local alone (every layer group, cold) with the configured sinks and
        with s = 0 (window only)."""
        torch, P = self.torch, self.P
        res = {}
        for name, zero in (("sinks", False), ("no_sinks", True)):
            calls = []
            for st in self.stacks:
                s_, w_ = st.local_args
                if zero:
                    s_ = 0
                ws = torch.zeros(max(256, P.attn_workspace_size(st.shape, s_, w_)), dtype=torch.uint8,
                                 device=self.dev)
                calls.append(P.prepare_local(st.shape, st.inp, s_, w_, st.out, st.lse, ws))
            res[f"{name}_us"] = self.kernel_time(calls, reps, cold=True)
        res["n_sink"] = max(st.local_args[0] for st in self.stacks)
        return res

    def read_ceiling(self, nbytes, reps=10):
        """Streaming-read ceiling: oda_stream_read over the first nbytes of the
        KV caches (cold), in GB/s."""
        torch, P = self.torch, self.P
        spans = []
        left = nbytes
        for st in self.stacks:
            for t in (st.k, st.v):
                take = min(left, t.numel() * t.element_size())
                take -= take % 16
                if take > 0:
                    spans.append((t, take))
                    left -= take
        calls = [P.prepare_stream_read(t, n, self.sink) for t, n in spans]
        done = nbytes - left
        us = self.kernel_time(calls, reps, cold=True)
        return dict(bytes=done, us=us, GBps=done / us / 1e3)

    def kernel_time(self, calls, reps, cold=True):
        """Mean duration (us) of one call bracketed by events on its stream."""
        torch = self.torch
        for c in calls:
            c()
        torch.cuda.synchronize()
        durs = []
        for _ in range(reps):
            if cold:
                self.flush()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for c in calls:
                c()
            b.record()
            torch.cuda.synchronize()
            durs.append(a.elapsed_time(b) * 1e3)
        return float(np.mean(durs))


TAU_MIN_GAP = 2 * FLAG_BORDER   # a threshold sits in a gap at least this wide between adjacent scores


def taus_for(scores, rhos):
    """Thresholds that flag round(rho * N) of the N scores: the midpoint of the
    gap between the m-th and (m+1)-th largest.  A gap narrower than
    TAU_MIN_GAP would leave the decisions on either side borderline, so the
    threshold moves to the nearest gap that is wide enough (the realised rate
    then differs from rho by that many decisions).  rho = 0 gives +inf, rho = 1
    gives -inf."""
    flat = np.sort(scores.reshape(-1))[::-1]
    N = len(flat)
    out = {}
    for rho in rhos:
        m = int(round(rho * N))
        if m <= 0:
            out[rho] = math.inf
            continue
        if m >= N:
            out[rho] = -math.inf
            continue
        wide = lambda i: 0 < i < N and flat[i - 1] - flat[i] >= TAU_MIN_GAP
        pick = m
        for off in range(N):
            if wide(m - off):
                pick = m - off
                break
            if wide(m + off):
                pick = m + off
                break
        out[rho] = float(0.5 * (flat[pick - 1] + flat[pick]))
    return out


def bytes_for(wl, seq, flagged_frac_per_step, head, gated_only=False):
    """Algorithmic bytes of one step: (Local, gate, per-request Full retry);
    gated_only restricts the retry to the gated layer groups."""
    from paper_2609_20734_amd import ledger as LG
    B = wl.batch
    local = sum(LG.attention_bytes(seq, *(st.local_sink, st.local_window) if st.gated else (0, st.native_window),
                                   st.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim)["total"]
                for st in wl.stacks)
    gate = LG.gate_bytes(head, B, wl.d_model, wl.d_hidden)["total"]
    full_all = [sum(LG.attention_bytes(seq, 0, st.native_window, st.num_layers, wl.num_q_heads, wl.num_kv_heads,
                                       wl.head_dim, requests=[b])["total"] for st in wl.stacks
                    if st.gated or not gated_only) for b in range(B)]
    return local, gate, full_all


# Host-side state of the CPU baseline, set before its process pool forks (the
# workers read it copy-on-write).
_CPU = {}


def _cpu_layer(i):
    """K and V of distinct cache layer i (a seeded N(0,1) bf16 slab tiled to
    the cache size: the oracle's work does not depend on the values)."""
    import oda_synth as S
    c = _CPU
    while len(c["k"]) <= i:
        j = len(c["k"])
        ks, vs = S.kv_cache_shapes(1, c["nb"], c["Hkv"], c["D"])
        slab_k = S.normal_bf16(S.rng(c["seed"] + j, S.STREAM_K), (1 << 20,))
        slab_v = S.normal_bf16(S.rng(c["seed"] + j, S.STREAM_V), (1 << 20,))
        c["k"].append(np.resize(slab_k, ks))
        c["v"].append(np.resize(slab_v, vs))
    return c["k"][i], c["v"][i]


def _cpu_task(task, branch):
    """Oracle time (s) of one (stack, layer, request) slice, Local or Full."""
    from oracle import attention as OA
    c = _CPU
    si, l, b = task
    s_, w_, native = c["stacks"][si]
    k, v = _cpu_layer(l % c["distinct"])
    if branch == "local":
        pos = (lambda n: OA.local_set(n, s_, w_)) if w_ > 0 else (lambda n: OA.native_window_set(n, native))
    else:
        pos = lambda n: OA.native_window_set(n, native)
    t0 = time.perf_counter()
    OA.decode_attention(c["q"][si][l:l + 1], k, v, c["table"], c["seq"], pos, c["scale"], requests=[b])
    return time.perf_counter() - t0


def _cpu_worker_init():
    from threadpoolctl import threadpool_limits
    _CPU["limits"] = threadpool_limits(limits=1)


def _cpu_local_task(task):
    return _cpu_task(task, "local")


def _cpu_full_task(task):
    return _cpu_task(task, "full")


def workload_seq_lens(wl, seed):
    import oda_synth as S
    if wl.seq_lens:
        return np.array(wl.seq_lens, dtype=np.int32)
    return S.uniform_seq_lens(seed, wl.batch, *wl.seq_range)


def cpu_baseline(wl, head, seed, rho, budget_s=10.0, mem_cap=8e9):
    """The fp64 oracle timed on the host on a bounded sample of the step, in
    two modes: (i) one thread (BLAS and OpenMP limited to 1) running the
    slices in turn; (ii) a process pool over (layer, request) slices, one
    single-threaded worker per core this process may use (at most 16).  Runs
    before the GPU is touched, so the pool's fork copies no GPU state.  Each
    slice is Local (or, for natively windowed layers, their window) or Full of
    one request in one layer; times are extrapolated to the whole step in
    attended positions, and the step weighs Full by rho (plus one gate
    evaluation for the batch)."""
    import multiprocessing as mp

    from threadpoolctl import threadpool_limits

    import oda_synth as S
    from oracle import attention as OA
    from oracle import gate as OG
    B, D, Hkv = wl.batch, wl.head_dim, wl.num_kv_heads
    seq = workload_seq_lens(wl, seed)
    mb = int(math.ceil(seq.max() / 16))
    table, nb = S.paged_block_table(S.rng(seed, S.STREAM_TABLE), seq, mb, permute=wl.permute)
    layer_bytes = 2 * nb * Hkv * D * 16 * 2
    _CPU.clear()
    _CPU.update(seed=seed, nb=nb, Hkv=Hkv, D=D, k=[], v=[], table=table, seq=seq, scale=1.0 / math.sqrt(D),
                distinct=max(1, min(sum(st.num_layers for st in wl.stacks), int(mem_cap // layer_bytes))),
                q=[S.normal_bf16(S.rng(seed + len(st.name), S.STREAM_Q), (st.num_layers, B, wl.num_q_heads, D))
                   for st in wl.stacks],
                stacks=[(st.local_sink if st.gated else 0, st.local_window if st.gated else 0, st.native_window)
                        for st in wl.stacks])
    tasks = [(si, l, b) for si, st in enumerate(wl.stacks) for l in range(st.num_layers) for b in range(B)]

    def positions(task, branch):
        si, _, b = task
        s_, w_, native = _CPU["stacks"][si]
        n = int(seq[b])
        if branch == "local" and w_ > 0:
            return len(OA.local_set(n, s_, w_))
        return len(OA.native_window_set(n, native))

    tot_local = sum(positions(t, "local") for t in tasks)
    tot_full = sum(positions(t, "full") for t in tasks)
    with threadpool_limits(limits=1):
        params = S.gate_params(seed, head, wl.d_model, wl.d_hidden)
        h, e, l_ = (x[0].astype(np.float64) for x in S.gate_inputs(seed, 1, B, wl.d_model))
        t0 = time.perf_counter()
        if head == "paper":
            OG.paper_head_score(params, wl.d_model, wl.d_hidden, 1e-6, h, e, l_)
        else:
            OG.mlp_score(params, wl.d_model, wl.d_hidden, l_)
        t_gate = time.perf_counter() - t0
        # (i) one thread
        t_loc = t_full = 0.0
        done = 0
        for t in tasks:
            _cpu_layer(t[1] % _CPU["distinct"])
            t_loc += _cpu_task(t, "local")
            t_full += _cpu_task(t, "full")
            done += 1
            if t_loc + t_full >= budget_s:
                break
    s_loc = sum(positions(t, "local") for t in tasks[:done])
    s_full = sum(positions(t, "full") for t in tasks[:done])
    one = t_gate + t_loc * tot_local / s_loc + rho * t_full * tot_full / s_full
    # (ii) process pool over (layer, request)
    cores = min(16, len(os.sched_getaffinity(0)))
    per_task = (t_loc + t_full) / done
    m = min(len(tasks), cores * max(1, int(budget_s / max(per_task, 1e-6))))
    for t in tasks[:m]:
        _cpu_layer(t[1] % _CPU["distinct"])
    ctx = mp.get_context("fork")
    with ctx.Pool(cores, initializer=_cpu_worker_init) as pool:
        pool.map(_cpu_local_task, tasks[:min(m, cores)])         # first touch of the workers
        t0 = time.perf_counter()
        pool.map(_cpu_local_task, tasks[:m], chunksize=1)
        w_loc = time.perf_counter() - t0
        t0 = time.perf_counter()
        pool.map(_cpu_full_task, tasks[:m], chunksize=1)
        w_full = time.perf_counter() - t0
    p_loc = sum(positions(t, "local") for t in tasks[:m])
    p_full = sum(positions(t, "full") for t in tasks[:m])
    pooled = t_gate + w_loc * tot_local / p_loc + rho * w_full * tot_full / p_full
    _CPU.clear()
    note = (f"K/V: seeded N(0,1) bf16 slabs tiled to the cache shape, {wl.batch} request(s), block table and "
            f"lengths as on the GPU; rho={rho} weighs Full; one gate evaluation ({head} head) for the batch")
    return dict(value=one * 1e6, unit="us/step", cores=1, kind="oracle", extrapolated=done < len(tasks),
                sample=f"{done} of {len(tasks)} (layer, request) slices, Local + Full, fp64 NumPy, 1 thread"
                       + (", extrapolated to every slice in attended positions" if done < len(tasks) else "")
                       + "; " + note,
                measured_s=t_gate + t_loc + t_full,
                host_cpus=os.cpu_count(), affinity_cpus=len(os.sched_getaffinity(0)),
                pool=dict(value=pooled * 1e6, unit="us/step", cores=cores, kind="oracle", extrapolated=m < len(tasks),
                          sample=f"{m} of {len(tasks)} slices over a {cores}-process pool (one thread each), "
                                 f"wall clock" + (", extrapolated to every slice in attended positions"
                                                  if m < len(tasks) else ""),
                          measured_s=w_loc + w_full))


def oracle_gate_scores(wl, seed, steps):
    """The fp64 oracle head's scores for every timed step's gate inputs (the
    same seeded buffers the GPU reads), per head kind: [steps][B].  Part of
    the CPU oracle leg (run before the GPU is touched); the sweep compares the
    kernel's flags at every operating point with the decisions these scores
    give."""
    import oda_synth as S
    from oracle import gate as OG
    h, e, l_ = (x.astype(np.float64).reshape(steps * wl.batch, wl.d_model)
                for x in S.gate_inputs(seed, steps, wl.batch, wl.d_model))
    out = {}
    for head in ("paper", "mlp"):
        params = S.gate_params(seed, head, wl.d_model, wl.d_hidden)
        if head == "paper":
            sc = OG.paper_head_score(params, wl.d_model, wl.d_hidden, 1e-6, h, e, l_)
        else:
            sc = OG.mlp_score(params, wl.d_model, wl.d_hidden, l_)
        out[head] = np.asarray(sc, dtype=np.float64).reshape(steps, wl.batch)
    return out


def flags_vs_oracle(gpu_flags, oracle_scores, tau, forced_np):
    """Kernel flags of the K steps against the oracle's decisions (Full iff
    score > tau, or the prescribed flag; nonfinite scores Full either way).
    Decisions of a threshold whose fp64 score lies within FLAG_BORDER of it
    are borderline: counted, and disagreements there reported apart."""
    score = oracle_scores
    fin = np.isfinite(score)
    if forced_np is None:
        want = (score > tau) | ~fin
        border = fin & (np.abs(score - tau) < FLAG_BORDER)
    else:
        want = (forced_np != 0) | ~fin
        border = np.zeros_like(want)
    differ = gpu_flags.astype(bool) != want
    return dict(decisions=int(want.size), borderline=int(border.sum()),
                flag_mismatch=int((differ & ~border).sum()), borderline_differ=int((differ & border).sum()))


def sweep_points(b, wl, args):
    """The configuration's operating points: recall rates set by the threshold
    (calibrated on this head's scores over the K steps) and Bernoulli schedules
    of forced flags (the gate still runs and is timed)."""
    import torch

    import oda_synth as S
    pts = []
    if wl.rhos:
        taus = taus_for(b.scores(), wl.rhos)
        pts += [dict(mode="tau", rho=r, tau=taus[r], forced=None, forced_np=None) for r in wl.rhos]
    for p in wl.bernoulli:
        f = S.bernoulli_flags(args.seed, b.K, wl.batch, p)
        pts.append(dict(mode="bernoulli", rho=p, tau=0.0, forced=torch.from_numpy(f).to(b.dev), forced_np=f))
    return pts


def primary_mode(wl):
    return "bernoulli" if wl.bernoulli else "tau"


def step_bytes(wl, b, pt, recalled, gated_only=False):
    local_b, gate_b, full_b = bytes_for(wl, b.seq_host, None, b.head, gated_only)
    _, _, full_all = bytes_for(wl, b.seq_host, None, b.head)
    K = b.K
    if pt["forced_np"] is None:
        full_part = recalled / (K * wl.batch) * sum(full_b)
    else:
        full_part = float(np.mean([(pt["forced_np"][t] * np.array(full_b)).sum() for t in range(K)]))
    return local_b + gate_b + full_part, sum(full_all)


def run_sweep(b, wl, args, full_us, gated_only=False, points=None):
    """Time the step at every operating point: `reps` repetitions of the K
    cold steps (the value is the median of the repetitions' means), then the
    same K steps warm (back to back, no flush).  The always-Full step is timed
    again after every point, and each point's ratio uses the mean of the
    always-Full times just before and just after it, so that drift of the
    machine's speed during a long run cancels."""
    K = b.K
    sweep = []
    full_before = getattr(b, "last_full_us", full_us)
    for pt in (points if points is not None else sweep_points(b, wl, args)):
        calls = b.step_calls(pt["tau"], forced=pt["forced"], gated_only=gated_only)
        reps = [b.timed(calls, args.warmup if i == 0 else 2, cold=True) for i in range(args.reps)]
        means = [r["us_mean"] for r in reps]
        per = np.concatenate([r["per_step"] for r in reps])
        us = float(np.median(means))
        recalled = reps[0]["recalled"]
        real = recalled / (K * wl.batch)
        nbytes, bytes_full = step_bytes(wl, b, pt, recalled, gated_only)
        full_after = b.timed(b.full_calls(), 2, cold=True)["us_mean"]
        full_adj = 0.5 * (full_before + full_after)
        full_before = b.last_full_us = full_after
        ent = dict(mode=pt["mode"], rho=pt["rho"], realised_rho=real, us=us, us_rep_min=min(means),
                   us_rep_max=max(means), us_step_median=float(np.median(per)), us_step_min=float(per.min()),
                   us_step_max=float(per.max()), GBps=nbytes / us / 1e3, full_adjacent_us=full_adj,
                   ratio=us / full_adj, ratio_first_full=us / full_us, ideal_ratio=nbytes / bytes_full)
        if pt["mode"] == "tau":
            ent["tau"] = pt["tau"]
        oracle = getattr(b, "oracle_scores", None)
        if oracle is not None:
            ent["flags_vs_oracle"] = flags_vs_oracle(b.step_flags(pt["tau"], pt["forced"]), oracle[b.head],
                                                     pt["tau"], pt["forced_np"])
        ent["hbm_frac"] = ent["GBps"] / HBM_PEAK_GBS
        ent["linearity"] = ent["ratio"] / ent["ideal_ratio"]
        if not args.no_warm:
            w = b.timed(calls, 2, cold=False)
            ent["warm_us"] = w["us_mean"]
            ent["warm_bracket_us"] = w["bracket_us"]
        sweep.append(ent)
        log(f"[bench] {b.head} head {pt['mode']} rho={pt['rho']:.3f} (real {real:.3f}) {us:.1f} us/step "
            f"ratio {ent['ratio']:.3f} ideal {ent['ideal_ratio']:.3f} x{ent['linearity']:.2f} {ent['GBps']:.0f} GB/s"
            + (" (retry on gated layers only)" if gated_only else "")
            + (f"; flags vs oracle: {ent['flags_vs_oracle']['flag_mismatch']} mismatched, "
               f"{ent['flags_vs_oracle']['borderline']} borderline of {ent['flags_vs_oracle']['decisions']}"
               if "flags_vs_oracle" in ent else ""))
    return sweep


def run_per_layer(b, wl, args, points):
    """The realism check: the same steps launched one layer per call, eager
    and as a captured HIP graph, against always-Full launched the same way."""
    fe, fg = b.per_layer_full(args.warmup)
    base = dict(eager_us=fe["us_mean"], graph_us=fg["us_mean"])
    log(f"[bench] per-layer always-Full: eager {fe['us_mean']:.1f} us/step, graph {fg['us_mean']:.1f} us/step")
    out = []
    for pt in points:
        eager, graph, branched = b.per_layer(pt["tau"], pt["forced"], args.warmup)
        ent = dict(mode=pt["mode"], rho=pt["rho"], realised_rho=eager["recalled"] / (b.K * wl.batch),
                   eager_us=eager["us_mean"], graph_us=graph["us_mean"], host_branch_us=branched["us_mean"],
                   graph_realised_rho=graph["recalled"] / (b.K * wl.batch),
                   eager_ratio=eager["us_mean"] / fe["us_mean"], graph_ratio=graph["us_mean"] / fg["us_mean"],
                   host_branch_ratio=branched["us_mean"] / fe["us_mean"])
        out.append(ent)
        log(f"[bench] per-layer launches rho={pt['rho']:.3f}: eager {eager['us_mean']:.1f} us/step, "
            f"graph {graph['us_mean']:.1f}, host branch {branched['us_mean']:.1f} "
            f"(x{ent['eager_ratio']:.3f} / x{ent['host_branch_ratio']:.3f} of per-layer always-Full)")
    return base, out


def gate_only(wl, args):
    """The recall gate alone, for counter profiling: both heads at the
    workload's batch and widths, ROOFLINE_REPS cold calls each (App. A.2 head
    first, then the MLP stand-in), then three 1 GiB copies for the counters'
    calibration.  Prints one JSON line with the calls' times and algorithmic
    bytes (fp32 weights + inputs + outputs, the ledger's)."""
    import torch

    import oda_synth as S
    import paper_2609_20734_amd as P
    from paper_2609_20734_amd import ledger as LG
    dev = torch.device("cuda:0")
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    B = wl.batch
    h, e, l_ = (torch.from_numpy(x[0]).to(dev) for x in S.gate_inputs(args.seed, 1, B, wl.d_model))
    score = torch.zeros(B, device=dev)
    flags = torch.zeros(B, dtype=torch.int32, device=dev)
    work = torch.zeros(B, dtype=torch.int32, device=dev)
    n_work = torch.zeros(1, dtype=torch.int32, device=dev)
    out = {}
    for head in ("paper", "mlp"):
        kind = P.HEAD_PAPER if head == "paper" else P.HEAD_MLP
        params = torch.from_numpy(S.gate_params(args.seed, head, wl.d_model, wl.d_hidden)).to(dev)
        g = P.gate_desc(kind, wl.d_model, wl.d_hidden, params, 1e-6)
        ws = torch.zeros(P.gate_workspace_size(g, B), dtype=torch.uint8, device=dev)
        call = P.prepare_gate(g, B, h, e, l_, 0.0, None, score, flags, work, n_work, None, ws)
        call()
        torch.cuda.synchronize()
        ts = []
        for _ in range(ROOFLINE_REPS):
            flush.max()
            a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            call()
            b_.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b_) * 1e3)
        out[head] = dict(us_per_call=float(np.median(ts)), bytes=LG.gate_bytes(head, B, wl.d_model, wl.d_hidden),
                         calls=1 + ROOFLINE_REPS)
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"gate_only": True, "workload": wl.name, "batch": B, "d_model": wl.d_model,
                      "d_hidden": wl.d_hidden, "heads": out, "copy_bytes": 1 << 30}), flush=True)


def extra_config(name, args):
    """A shortened run of another workload in the same process: the always-Full
    step, the threshold (and Bernoulli) sweep of the App. A.2 head with each
    point's flags checked against the fp64 oracle head, and the roofline
    launch with its counter traffic.  No warm timing, per-layer mode, decode
    loop or second head."""
    import copy

    import torch

    from paper_2609_20734_amd import workloads as WL
    wl = WL.ALL[name]
    K = wl.steps
    oracle = oracle_gate_scores(wl, args.seed, K)
    b = Bench(wl, "paper", args.seed, K, local="paged" if args.local_paged else "ring")
    b.oracle_scores = oracle
    sub = copy.copy(args)
    sub.no_warm = True
    fulls = [b.timed(b.full_calls(), args.warmup if i == 0 else 2, cold=True) for i in range(args.reps)]
    full_us = float(np.median([f["us_mean"] for f in fulls]))
    sweep = run_sweep(b, wl, sub, full_us)
    local_b, gate_b, full_b = bytes_for(wl, b.seq_host, None, "paper")
    bytes_full = sum(full_b)
    t = b.kernel_time(b.full_calls()[0], reps=ROOFLINE_REPS, cold=True)
    ceil_full = b.read_ceiling(bytes_full)
    roof = dict(bound="hbm", achieved=bytes_full / t / 1e3, peak=HBM_PEAK_GBS, unit="GB/s",
                traffic=measured_traffic(wl.name, bytes_full), bytes_per_launch=bytes_full, us_per_launch=t,
                read_ceiling_GBps=ceil_full["GBps"])
    roof["frac"] = roof["achieved"] / roof["peak"]
    out = dict(workload=f"{wl.name}: {wl.num_layers} layers, B={wl.batch}, {wl.num_q_heads}q/{wl.num_kv_heads}kv heads, "
                        f"D={wl.head_dim}, n={'/'.join(str(x) for x in sorted(set(b.seq_host.tolist()))[:4])}, "
                        f"W={wl.stacks[-1].local_window}, s={wl.stacks[-1].local_sink}, Local from the "
                        f"{'paged cache' if args.local_paged else 'direct-ring workspace'}, paper recall head "
                        f"{wl.d_model}->{wl.d_hidden}->1, cold",
               steps=K, reps=args.reps, always_full_us=round(full_us, 3),
               sweep=[rounded(e) for e in sweep], roofline=rounded(roof))
    del b
    torch.cuda.empty_cache()
    return out


def rounded(d, nd=4):
    return {k: (round(v, nd) if isinstance(v, float) else v) for k, v in d.items()}


PAPER_LENGTHS = (4139, 15918, 31400, 63852, 128852, 261696, 516788)


def decoder_bench(args):
    """Tokens/s of whole decode steps (Alg. 1 with the commit of App. A.5) on a
    synthetic Qwen3-1.7B-shaped decoder at batch one, per context length:
    native Full, standalone Local, ODA with a prescribed schedule (the first
    2 / 4 / 8 of every 16 steps Full, App. B.7; the recall head still runs
    every step).  Each step is launched as HIP graphs: ODA replays its local
    stage, reads the device's count of flagged requests into pinned host
    memory (one host synchronisation per step, the branch of Alg. 1), replays
    the Full-retry stage only if that count is nonzero, then the output stage
    (also timed: one graph per step with the retry stage always replayed,
    whose kernels exit early when nothing is flagged)."""
    import torch

    import oda_synth as S
    import paper_2609_20734_amd as P
    from paper_2609_20734_amd import decoder as PD

    dev = torch.device("cuda:0")
    shape = PD.QWEN3_1_7B
    L, d, Hq, Hkv, D = shape.num_layers, shape.d_model, shape.num_q_heads, shape.num_kv_heads, shape.head_dim
    lengths = [int(x) for x in args.lengths.split(",")] if args.lengths else list(PAPER_LENGTHS)
    warm, T, period = 16, args.decoder_steps, 16
    n_sink, window = 4, 2048
    margin = warm + T + 16
    cap_blocks = int(math.ceil((max(lengths) + margin) / 16))
    kv_bytes = 2 * L * cap_blocks * Hkv * D * 16 * 2
    free, _ = torch.cuda.mem_get_info()
    log(f"[decoder] Qwen3-1.7B shape, weights {shape.weight_bytes() / 1e9:.2f} GB/forward, KV {kv_bytes / 1e9:.1f} GB, "
        f"free {free / 1e9:.1f} GB")
    if kv_bytes + 8e9 > free:
        raise SystemExit("not enough device memory for the longest context")
    w = S.decoder_weights_device(args.seed, L, d, Hq, Hkv, D, shape.d_ffn, shape.vocab, dev)
    k_cache = torch.empty((L, cap_blocks, Hkv, D // 8, 16, 8), dtype=torch.bfloat16, device=dev)
    v_cache = torch.empty((L, cap_blocks, Hkv, D, 16), dtype=torch.bfloat16, device=dev)
    for i, t in enumerate((k_cache, v_cache)):
        for l in range(L):
            S.fill_normal_bf16_(t[l], args.seed + 31 * l, S.STREAM_K + i)
            if l % 7 == 6:
                torch.cuda.synchronize()
                log(f"[decoder] filled {'KV'[i]} cache layers 0..{l}")
    dt = 1024                                        # App. A.2 head for d = 2048: 28,325,889 parameters
    gparams = torch.from_numpy(S.gate_params(args.seed, "paper", d, dt)).to(dev)
    gate = P.gate_desc(P.HEAD_PAPER, d, dt, gparams, 1e-6)
    cont = torch.from_numpy(S.tokens(args.seed, warm + T, 1, shape.vocab)).to(dev)
    n_host = torch.zeros(1, dtype=torch.int32).pin_memory()
    results = []
    for n in lengths:
        nblk = int(math.ceil((n + margin) / 16))
        perm = S.rng(args.seed + n, S.STREAM_TABLE).permutation(cap_blocks)[:nblk].astype(np.int32)
        table = torch.from_numpy(perm[None, :]).to(dev)
        seq0 = torch.tensor([n + 1], dtype=torch.int32, device=dev)     # prompt of n tokens + the current one
        seq = seq0.clone()
        dec = PD.Decoder(shape, w, 1, k_cache, v_cache, table, seq, nblk, n + margin, cap_blocks, n_sink, window,
                         gate=gate, tau=0.0, prescribed=True)
        row = {"input_tokens": n}

        def capture(i_stage, make):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for c in make()[i_stage]:
                    c()
            return g

        def capture_all(make):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for st in make():
                    for c in st:
                        c()
            return g

        def timed(step_fn, sched):
            seq.copy_(seq0)
            dec.counter.zero_()
            torch.cuda.synchronize()
            for t in range(warm):
                step_fn(t, sched)
            torch.cuda.synchronize()
            seq.copy_(seq0)
            dec.counter.zero_()
            a, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            for t in range(T):
                step_fn(warm + t, sched)
            b_.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b_) / 1e3, int(dec.counter.item())

        def set_inputs(t, sched):
            dec.tokens.copy_(cont[t])
            if sched is not None:
                dec.forced.copy_(sched[t % period])

        for name, make in (("full", dec.full_stages), ("local", dec.local_stages)):
            g = capture_all(make)

            def step(t, sched, g=g):
                set_inputs(t, None)
                g.replay()
            secs, _ = timed(step, None)
            row[f"{name}_tps"] = T / secs
            del g
        g_loc, g_retry, g_out = (capture(i, dec.oda_stages) for i in range(3))
        g_all = capture_all(dec.oda_stages)
        for k in (2, 4, 8):
            sched = torch.from_numpy(S.periodic_schedule(period, k).astype(np.int32).reshape(period, 1)).to(dev)

            def step_host(t, sched):
                set_inputs(t, sched)
                g_loc.replay()
                n_host.copy_(dec.n_work, non_blocking=True)
                torch.cuda.current_stream().synchronize()
                if int(n_host[0]) > 0:
                    g_retry.replay()
                g_out.replay()

            def step_dev(t, sched):
                set_inputs(t, sched)
                g_all.replay()
            secs, rec = timed(step_host, sched)
            row[f"oda{k}_tps"] = T / secs
            row[f"oda{k}_full_calls"] = rec
            secs, rec2 = timed(step_dev, sched)
            row[f"oda{k}_device_only_tps"] = T / secs
            assert rec == rec2 == k * T // period, (rec, rec2)
        del g_loc, g_retry, g_out, g_all
        for key in list(row):
            if key.endswith("_tps"):
                row[key] = round(row[key], 2)
        for k in (2, 4, 8):
            row[f"oda{k}_speedup"] = round(row[f"oda{k}_tps"] / row["full_tps"], 3)
        row["local_speedup"] = round(row["local_tps"] / row["full_tps"], 3)
        log(f"[decoder] n={n}: Full {row['full_tps']:.1f} tok/s, Local {row['local_tps']:.1f}, "
            + ", ".join(f"ODA {100 * k // 16}% {row[f'oda{k}_tps']:.1f} (x{row[f'oda{k}_speedup']:.2f}; "
                        f"device-only {row[f'oda{k}_device_only_tps']:.1f})" for k in (2, 4, 8)))
        results.append(row)
        del dec
    print(json.dumps({"decoder": {"model": "Qwen3-1.7B-shaped synthetic decoder (28 x 2048, 16q/8kv x 128, "
                                           "SwiGLU 6144, vocab 151936, bf16 weights)",
                                  "batch": 1, "local": {"sinks": n_sink, "window": window},
                                  "recall_head": "App. A.2, 2048 -> 1024", "steps": T, "warmup": warm,
                                  "weight_bytes_per_forward": shape.weight_bytes(), "rows": results}}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0, help="timed steps per repetition (default: the workload's)")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--reps", type=int, default=3, help="repetitions of the K steps per operating point")
    ap.add_argument("--config", default="mixed",
                    help="workload (default: the batched mixed-length stack, the largest single-GPU configuration)")
    ap.add_argument("--head", default="paper", choices=["paper", "mlp"])
    ap.add_argument("--seed", type=int, default=1234)
    ap.add_argument("--split-blocks", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-warm", action="store_true", help="skip the warm (back-to-back) timing of each point")
    ap.add_argument("--one-head", action="store_true", help="skip the second recall head's sweep")
    ap.add_argument("--no-per-layer", action="store_true", help="skip the per-layer launch mode")
    ap.add_argument("--no-loop", action="store_true", help="skip the growing-context decode loop (graph) section")
    ap.add_argument("--loop-only", action="store_true", help="only the decode loop section (for profiling)")
    ap.add_argument("--decoder", action="store_true",
                    help="time whole steps of the synthetic decoder (tokens/s) instead of the attention path")
    ap.add_argument("--lengths", default="", help="--decoder: comma-separated context lengths")
    ap.add_argument("--decoder-steps", type=int, default=64, help="--decoder: timed steps per method")
    ap.add_argument("--local-paged", action="store_true",
                    help="Local reads the paged cache through the block table instead of the direct-ring workspace")
    ap.add_argument("--extra-configs", default="llama3-8b,long,hybrid",
                    help="comma-separated workloads given a shortened run after the main one ('' for none)")
    ap.add_argument("--gate-only", action="store_true",
                    help="only the recall gate (both heads) plus a 1 GiB copy, for PMC profiling")
    ap.add_argument("--roofline-only", action="store_true",
                    help="only the counter legs (Local, empty Full, the roofline Full launch) plus a 1 GiB copy, "
                         "for PMC profiling")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    if args.decoder:
        decoder_bench(args)
        return

    from paper_2609_20734_amd import workloads as WL
    wl = WL.ALL[args.config]
    if args.gate_only:
        gate_only(wl, args)
        return
    K = args.steps if args.steps > 0 else wl.steps
    args.reps = max(1, args.reps)
    pts_nominal = list(wl.bernoulli) if wl.bernoulli else list(wl.rhos)
    head_rho = min(pts_nominal, key=lambda r: abs(r - HEADLINE_RHO)) if pts_nominal else 1.0

    # the CPU oracle leg first: its process pool forks before the GPU is touched;
    # it also scores every timed step's gate inputs with the fp64 oracle head
    cb = None
    oracle_scores = None
    if not (args.no_cpu_baseline or args.roofline_only or args.loop_only):
        cb = cpu_baseline(wl, args.head, args.seed, head_rho)
        log(f"[bench] CPU oracle: {cb['value'] / 1e3:.1f} ms/step on 1 thread, {cb['pool']['value'] / 1e3:.1f} ms/step "
            f"on {cb['pool']['cores']} processes (host: {cb['host_cpus']} CPUs, {cb['affinity_cpus']} usable)")
        oracle_scores = oracle_gate_scores(wl, args.seed, K)

    import torch
    b = Bench(wl, args.head, args.seed, K, args.split_blocks,
              growth=0 if (args.no_loop or args.roofline_only) else 16 * 8,
              local="paged" if args.local_paged else "ring")
    P = b.P
    b.oracle_scores = oracle_scores
    local_b, gate_b, full_b = bytes_for(wl, b.seq_host, None, args.head)
    bytes_full = sum(full_b)

    if args.roofline_only:
        # dispatch order (the counter summaries rely on it): 1 + R Local launches,
        # 1 + R empty Full launches (list of zero requests), 1 + R roofline
        # launches (Full over every request), then three 1 GiB copies
        t_loc = b.kernel_time([b.local_call(s) for s in b.stacks], reps=ROOFLINE_REPS, cold=True)
        b.n_work.zero_()
        t_empty = b.kernel_time([P.prepare_full(s.shape, s.inp, s.stack.native_window, None, b.work, b.n_work,
                                                s.out, s.lse, s.ws_full) for s in b.stacks],
                                reps=ROOFLINE_REPS, cold=True)
        t = b.kernel_time(b.full_calls()[0], reps=ROOFLINE_REPS, cold=True)
        src = torch.ones(1 << 28, dtype=torch.float32, device=b.dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)          # calibration: 1 GiB read + 1 GiB written
        torch.cuda.synchronize()
        print(json.dumps({"roofline_only": True, "kernel": ROOFLINE_KERNEL, "us_per_launch": t,
                          "bytes_per_launch": bytes_full, "reps": ROOFLINE_REPS, "local_us": t_loc,
                          "local_bytes": local_b, "empty_full_us": t_empty,
                          "copy_bytes": 1 << 30, "source_sha256": source_sha256()}), flush=True)
        return

    if args.loop_only:
        print(json.dumps({"decode_loop": b.decode_loop()}), flush=True)
        return

    # always-Full baseline
    fulls = [b.timed(b.full_calls(), args.warmup if i == 0 else 2, cold=True) for i in range(args.reps)]
    full_us = float(np.median([f["us_mean"] for f in fulls]))
    log(f"[bench] always-Full {full_us:.1f} us/step ({bytes_full / full_us / 1e3:.0f} GB/s)")

    # operating points with the App. A.2 head (headline), then the MLP stand-in
    head0 = args.head
    pts = sweep_points(b, wl, args)
    sweep = run_sweep(b, wl, args, full_us, points=pts)
    primary = [p for p in pts if p["mode"] == primary_mode(wl)]
    gated_only = []
    if any(not st.gated for st in wl.stacks):
        gated_only = run_sweep(b, wl, args, full_us, gated_only=True, points=primary)
    per_layer_full, per_layer = (None, []) if args.no_per_layer else run_per_layer(b, wl, args, primary)
    other = "mlp" if head0 == "paper" else "paper"
    sweep_other = []
    if not args.one_head:
        b.set_head(other)
        sweep_other = run_sweep(b, wl, args, full_us)
        b.set_head(head0)

    loop = [] if args.no_loop else b.decode_loop()
    layout = b.local_layout()
    log(f"[bench] Local alone, cold: permuted block table {layout['permuted_us']:.1f} us, "
        f"contiguous table {layout['contiguous_us']:.1f} us, direct ring {layout['ring_us']:.1f} us "
        f"(rings {layout['ring_bytes'] / 1e9:.2f} GB); one layer: permuted {layout['one_layer_permuted_us']:.2f} us, "
        f"ring {layout['one_layer_ring_us']:.2f} us")
    sinks = b.local_sinks()
    log(f"[bench] Local alone, cold: s={sinks['n_sink']} {sinks['sinks_us']:.1f} us, s=0 {sinks['no_sinks_us']:.1f} us")

    # roofline of the dominant kernel: the Full split-K pass over every request
    # (one launch of attn_split_kernel<128, false>; no merge launch at this size),
    # the last ROOFLINE_REPS dispatches of that kernel in this process
    fcalls = b.full_calls()[0]
    t_full_call = b.kernel_time(fcalls, reps=ROOFLINE_REPS, cold=True)
    ceil_full = b.read_ceiling(bytes_full)
    ceil_local = b.read_ceiling(local_b)
    log(f"[bench] streaming-read ceiling: {ceil_full['GBps']:.0f} GB/s over {ceil_full['bytes'] / 1e9:.2f} GB, "
        f"{ceil_local['GBps']:.0f} GB/s over {ceil_local['bytes'] / 1e6:.0f} MB")
    roof = dict(bound="hbm", achieved=bytes_full / t_full_call / 1e3, peak=HBM_PEAK_GBS, unit="GB/s",
                traffic=measured_traffic(wl.name, bytes_full))
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = ROOFLINE_KERNEL + " (oda_full_decode_attn, every request)"
    roof["bytes_per_launch"] = bytes_full
    roof["us_per_launch"] = t_full_call
    roof["read_ceiling_GBps"] = ceil_full["GBps"]
    roof["frac_of_read_ceiling"] = roof["achieved"] / ceil_full["GBps"]

    prim = [e for e in sweep if e["mode"] == primary_mode(wl)]
    head_ent = min(prim, key=lambda e: abs(e["rho"] - HEADLINE_RHO)) if prim else None
    value = head_ent["us"] if head_ent else full_us
    nset = sorted(set(b.seq_host.tolist()))
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "us/step", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "reps": args.reps, "ms_per_step": round(value / 1e3, 6), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.num_layers} layers, B={wl.batch}, {wl.num_q_heads}q/{wl.num_kv_heads}kv "
                               f"heads, D={wl.head_dim}, "
                               + (f"n~U[{wl.seq_range[0]},{wl.seq_range[1]}] (seeded; realised mean "
                                  f"{float(b.seq_host.mean()):.0f}, KV {sum(full_b) / 1e9:.1f} GB)"
                                  if wl.seq_range else f"n={'/'.join(str(x) for x in nset[:4])}"
                                  f"{'...' if len(nset) > 4 else ''}") + ", "
                               f"W={wl.stacks[-1].local_window}, s={wl.stacks[-1].local_sink}, paged bf16 KV "
                               f"(block 16, permuted), Local from the "
                               f"{'paged cache' if args.local_paged else 'direct-ring workspace'}, "
                               f"{args.head} recall head {wl.d_model}->{wl.d_hidden}->1, "
                               f"{head_ent['mode'] + ' ' if head_ent else ''}rho={head_ent['rho'] if head_ent else 1.0}, "
                               f"cold (Infinity Cache flushed between steps)",
                   "head": args.head, "seed": args.seed, "split_blocks": args.split_blocks,
                   "local": "paged" if args.local_paged else "ring"},
        "GBps": round(head_ent["GBps"], 1) if head_ent else None,
        "always_full_us": round(full_us, 3),
        "always_full_us_reps": [round(f["us_mean"], 3) for f in fulls],
        "always_full_GBps": round(bytes_full / full_us / 1e3, 1),
        "sweep": [rounded(e) for e in sweep],
        f"sweep_{other}_head": [rounded(e) for e in sweep_other],
        "per_layer": [rounded(e, 3) for e in per_layer],
        "per_layer_always_full": rounded(per_layer_full, 3) if per_layer_full else None,
        "decode_loop": [rounded(e, 3) for e in loop],
        "local_window_layout": rounded(layout, 3),
        "local_sinks": rounded(sinks, 3),
        "read_ceiling": {"full_size": rounded(ceil_full, 3), "local_size": rounded(ceil_local, 3)},
        "roofline": rounded(roof),
    }
    if gated_only:
        res["sweep_gated_only"] = [rounded(e) for e in gated_only]
    extras = [c for c in args.extra_configs.split(",") if c and c != wl.name]
    if extras:
        del b
        torch.cuda.empty_cache()
        res["extra_configs"] = {}
        for c in extras:
            res["extra_configs"][c] = extra_config(c, args)
            e = res["extra_configs"][c]
            log(f"[bench] {c}: always-Full {e['always_full_us']:.1f} us/step, roofline "
                f"{e['roofline']['frac']:.3f} of 8 TB/s; " + ", ".join(
                    f"rho={p['rho']}: {p['us']:.1f} us x{p['linearity']:.2f}" for p in e["sweep"]))
    if cb is not None:
        cbr = rounded(cb, 3)
        cbr["pool"] = rounded(cb["pool"], 3)
        res["cpu_baseline"] = cbr
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
