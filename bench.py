#!/usr/bin/env python3
"""Benchmark of the ODA decode-step hot path on one MI355X.

A step is one pass of the whole path over one batch: Local decode attention
for every layer and request, the recall gate (score + device predicate +
compaction), and Full decode attention for the flagged requests only, all on
one stream.  The recall rate rho is swept by the threshold tau (calibrated on
the gate's scores over the K timed steps), and compared against the
always-Full baseline (Full for every request, no Local, no gate).

Timing: every step is bracketed by HIP events on the stream the library
launches on.  Headline ("cold") numbers read a 1 GiB scratch buffer between
steps, outside the events, so the 256 MB Infinity Cache holds no KV or gate
weights at the start of a step; "warm" numbers run the K steps back to back.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config llama3-8b] [--head paper|mlp]

Prints one JSON line: the headline value (µs per step at the recall rate
nearest 0.1), the per-rate sweep for both recall heads, the decode loop, the
roofline of the dominant kernel and the CPU oracle baseline.

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
ROOFLINE_REPS = 20
ROOFLINE_KERNEL = "attn_split_kernel<128, false>"
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_20734_amd", "csrc", "attention.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "full_split_llama3-8b_traffic.txt")


def source_sha256() -> str:
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per launch of the roofline kernel from the committed PMC summary,
    or None if there is none or the kernel source changed since it was taken."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha256():
        return None
    try:
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
        self.ws_local = torch.empty(P.attn_workspace_size(self.shape, loc_s, loc_w), dtype=torch.uint8, device=dev)
        self.ws_full = torch.empty(P.attn_workspace_size(self.shape, 0, stack.native_window), dtype=torch.uint8,
                                   device=dev)


class Bench:
    def __init__(self, wl, head, seed, steps, split_blocks=0, growth=0):
        import torch

        import oda_synth as S
        import paper_2609_20734_amd as P
        self.P, self.torch, self.wl, self.seed, self.K = P, torch, wl, seed, steps
        dev = torch.device("cuda:0")
        self.dev = dev
        B = wl.batch
        if wl.seq_lens:
            seq = np.array(wl.seq_lens, dtype=np.int32)
        else:
            seq = S.uniform_seq_lens(seed, B, *wl.seq_range)
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
        # 1 GiB read between steps evicts the 256 MB Infinity Cache with clean lines
        # (a write flush would leave dirty lines for the next step to write back)
        self.flush_buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)

    def flush(self):
        self.flush_buf.max()

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
        self.ws_gate = torch.empty(P.gate_workspace_size(self.gate, wl.batch), dtype=torch.uint8, device=self.dev)

    # -- calls ---------------------------------------------------------------
    def step_calls(self, tau, forced=None):
        """Per step t: the list of pre-marshalled calls of one decode step."""
        P = self.P
        local = [P.prepare_local(s.shape, s.inp, *s.local_args, s.out, s.lse, s.ws_local) for s in self.stacks]
        full = [P.prepare_full(s.shape, s.inp, s.stack.native_window, None, self.work, self.n_work, s.out, s.lse,
                               s.ws_full) for s in self.stacks]
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
        res = []

        def one_period(forced):
            for t in range(period):
                for st, (kl, vl, kf, vf) in zip(self.stacks, cands):
                    inp = P.inputs(st.q, st.k, st.v, self.dtable, self.dseq, scale, kl[t], vl[t])
                    P.local_decode_attn(st.shape, inp, *st.local_args, st.out, st.lse, st.ws_local)
                P.recall_gate(self.gate, B, self.h[t % self.K], self.e[t % self.K], self.l[t % self.K], 0.0,
                              forced[t], self.score, self.flags, self.work, self.n_work, self.counter, self.ws_gate)
                for st, (kl, vl, kf, vf) in zip(self.stacks, cands):
                    inp = P.inputs(st.q, st.k, st.v, self.dtable, self.dseq, scale, kf[t], vf[t])
                    P.full_decode_attn(st.shape, inp, st.stack.native_window, None, self.work, self.n_work,
                                       st.out, st.lse, st.ws_full)
                for i, (st, (kl, vl, kf, vf)) in enumerate(zip(self.stacks, cands)):
                    P.commit_kv(st.shape, st.k, st.v, self.dtable, self.dseq, kl[t], vl[t], kf[t], vf[t],
                                self.flags, i == len(self.stacks) - 1)

        for k in firsts:
            sched = np.stack([S.periodic_schedule(period, k)] * B, axis=1).astype(np.int32)
            forced = torch.from_numpy(sched).to(self.dev)
            # eager: launched from the host every period
            self.dseq.copy_(seq0)
            one_period(forced)
            torch.cuda.synchronize()
            self.dseq.copy_(seq0)
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
            self.dseq.copy_(seq0)
            g = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                one_period(forced)
            self.dseq.copy_(seq0)
            g.replay()
            torch.cuda.synchronize()
            self.dseq.copy_(seq0)
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
        self.dseq.copy_(seq0)
        return res

    def full_calls(self):
        P = self.P
        full = [P.prepare_full(s.shape, s.inp, s.stack.native_window, None, None, None, s.out, s.lse, s.ws_full)
                for s in self.stacks]
        return [full] * self.K

    def scores(self):
        """Gate scores of all K steps (tau = +inf), for threshold calibration."""
        out = np.zeros((self.K, self.wl.batch))
        for t in range(self.K):
            self.P.recall_gate(self.gate, self.wl.batch, self.h[t], self.e[t], self.l[t], math.inf, None,
                               self.score, self.flags, None, None, None, self.ws_gate)
            out[t] = self.score.cpu().numpy()
        return out

    # -- timing --------------------------------------------------------------
    def timed(self, steps, warmup, cold=True):
        torch = self.torch
        for t in range(warmup):
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
        the permuted block table and through a contiguous one (identity table,
        same cache, same lengths): the cost of scattered paged-window reads,
        which decides whether a contiguous ring workspace for Local would pay."""
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
        return res

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


def taus_for(scores, rhos):
    flat = np.sort(scores.reshape(-1))[::-1]
    N = len(flat)
    out = {}
    for rho in rhos:
        m = int(round(rho * N))
        if m <= 0:
            out[rho] = math.inf
        elif m >= N:
            out[rho] = -math.inf
        else:
            out[rho] = float(0.5 * (flat[m - 1] + flat[m]))
    return out


def bytes_for(wl, seq, flagged_frac_per_step, head):
    """Average algorithmic bytes per step given the realised per-step flag sets."""
    from paper_2609_20734_amd import ledger as LG
    B = wl.batch
    local = sum(LG.attention_bytes(seq, *(st.local_sink, st.local_window) if st.gated else (0, st.native_window),
                                   st.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim)["total"]
                for st in wl.stacks)
    gate = LG.gate_bytes(head, B, wl.d_model, wl.d_hidden)["total"]
    full_all = [sum(LG.attention_bytes(seq, 0, st.native_window, st.num_layers, wl.num_q_heads, wl.num_kv_heads,
                                       wl.head_dim, requests=[b])["total"] for st in wl.stacks) for b in range(B)]
    return local, gate, full_all


def cpu_baseline(b, rho, budget_s=15.0):
    """The fp64 oracle timed on a bounded sample of the same step, 1 thread."""
    from threadpoolctl import threadpool_limits

    from oracle import attention as OA
    from oracle import gate as OG
    wl = b.wl
    st = b.stacks[-1]
    L = st.stack.num_layers
    seq = b.seq_host
    with threadpool_limits(limits=1):
        # gate (one step)
        t0 = time.perf_counter()
        params = b.params.cpu().numpy()
        h, e, l = (x[0].cpu().numpy().astype(np.float64) for x in (b.h, b.e, b.l))
        if b.head == "paper":
            OG.paper_head_score(params, wl.d_model, wl.d_hidden, 1e-6, h, e, l)
        else:
            OG.mlp_score(params, wl.d_model, wl.d_hidden, l)
        t_gate = time.perf_counter() - t0
        # per layer: copy the layer's cache once, then Local and Full for every request
        q_all = b.stacks[-1].q.cpu().numpy().view(np.uint16)
        table = b.dtable.cpu().numpy()
        t_local = t_full = 0.0
        layers = 0
        for layer in range(L):
            kl = st.k[layer:layer + 1].cpu().view(b.torch.int16).numpy().view(np.uint16)
            vl = st.v[layer:layer + 1].cpu().view(b.torch.int16).numpy().view(np.uint16)
            ql = q_all[layer:layer + 1]
            s_, w_ = st.local_args
            t0 = time.perf_counter()
            OA.decode_attention(ql, kl, vl, table, seq, lambda n: OA.local_set(n, s_, w_), 1 / math.sqrt(wl.head_dim))
            t1 = time.perf_counter()
            OA.decode_attention(ql, kl, vl, table, seq, lambda n: OA.native_window_set(n, st.stack.native_window),
                                1 / math.sqrt(wl.head_dim))
            t2 = time.perf_counter()
            t_local += t1 - t0
            t_full += t2 - t1
            layers += 1
            if t_local + t_full + t_gate > budget_s:
                break
    scale = wl.num_layers / layers
    per_step = t_gate + scale * (t_local + rho * t_full)
    return dict(value=per_step * 1e6, unit="us/step", cores=1, kind="oracle",
                sample=f"{layers} of {wl.num_layers} layers (Local + Full, all {wl.batch} requests) and one gate "
                       f"evaluation, fp64 NumPy, 1 thread; extrapolated linearly to {wl.num_layers} layers at "
                       f"rho={rho} (Full time weighted by rho)",
                measured_s=t_gate + t_local + t_full)


def run_sweep(b, wl, args, full_us):
    """Time the step over the configuration's recall rates (threshold-driven) or
    Bernoulli schedules (forced flags, gate still run); one entry per point."""
    import torch
    K = b.K
    local_b, gate_b, full_b = bytes_for(wl, b.seq_host, None, b.head)
    bytes_full = sum(full_b)
    sweep = []
    if wl.rhos:
        sc = b.scores()
        taus = taus_for(sc, wl.rhos)
        points = [(rho, taus[rho], None, None) for rho in wl.rhos]
    else:
        import oda_synth as S
        points = []
        for p in wl.bernoulli:
            forced_np = S.bernoulli_flags(args.seed, K, wl.batch, p)
            points.append((p, 0.0, torch.from_numpy(forced_np).to(b.dev), forced_np))
    for rho, tau, forced, forced_np in points:
        r = b.timed(b.step_calls(tau, forced=forced), args.warmup, cold=True)
        real = r["recalled"] / (K * wl.batch)
        if forced_np is None:
            full_part = real * bytes_full
        else:
            full_part = float(np.mean([(forced_np[t] * np.array(full_b)).sum() for t in range(K)]))
        step_bytes = local_b + gate_b + full_part
        ent = dict(rho=rho, realised_rho=real, us=r["us_mean"], us_median=r["us_median"], us_min=r["us_min"],
                   us_max=r["us_max"], GBps=step_bytes / r["us_mean"] / 1e3, ratio=r["us_mean"] / full_us,
                   ideal_ratio=step_bytes / bytes_full)
        if forced_np is None:
            ent["tau"] = tau
        ent["hbm_frac"] = ent["GBps"] / HBM_PEAK_GBS
        ent["linearity"] = ent["ratio"] / ent["ideal_ratio"]
        if args.warm:
            w = b.timed(b.step_calls(tau, forced=forced), args.warmup, cold=False)
            ent["warm_us"] = w["us_mean"]
            ent["warm_bracket_us"] = w["bracket_us"]
        sweep.append(ent)
        log(f"[bench] {b.head} head rho={rho:.3f} (real {real:.3f}) {r['us_mean']:.1f} us/step ratio {ent['ratio']:.3f} "
            f"ideal {ent['ideal_ratio']:.3f} x{ent['linearity']:.2f} {ent['GBps']:.0f} GB/s")
    return sweep


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
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="llama3-8b")
    ap.add_argument("--head", default="paper", choices=["paper", "mlp"])
    ap.add_argument("--seed", type=int, default=1234)
    ap.add_argument("--split-blocks", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--warm", action="store_true", help="also time back-to-back (warm) steps")
    ap.add_argument("--one-head", action="store_true", help="skip the second recall head's sweep")
    ap.add_argument("--no-loop", action="store_true", help="skip the growing-context decode loop (graph) section")
    ap.add_argument("--loop-only", action="store_true", help="only the decode loop section (for profiling)")
    ap.add_argument("--decoder", action="store_true",
                    help="time whole steps of the synthetic decoder (tokens/s) instead of the attention path")
    ap.add_argument("--lengths", default="", help="--decoder: comma-separated context lengths")
    ap.add_argument("--decoder-steps", type=int, default=64, help="--decoder: timed steps per method")
    ap.add_argument("--roofline-only", action="store_true",
                    help="only the roofline leg (always-Full calls) plus a 1 GiB copy, for PMC profiling")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    if args.decoder:
        decoder_bench(args)
        return

    import torch

    from paper_2609_20734_amd import workloads as WL
    wl = WL.ALL[args.config]
    K = args.steps
    b = Bench(wl, args.head, args.seed, K, args.split_blocks,
              growth=0 if (args.no_loop or args.roofline_only) else 16 * 8)
    P = b.P
    local_b, gate_b, full_b = bytes_for(wl, b.seq_host, None, args.head)
    bytes_full = sum(full_b)

    if args.roofline_only:
        t = b.kernel_time(b.full_calls()[0], reps=ROOFLINE_REPS, cold=True)
        src = torch.ones(1 << 28, dtype=torch.float32, device=b.dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)          # calibration: 1 GiB read + 1 GiB written
        torch.cuda.synchronize()
        print(json.dumps({"roofline_only": True, "kernel": ROOFLINE_KERNEL, "us_per_launch": t,
                          "bytes_per_launch": bytes_full, "reps": ROOFLINE_REPS,
                          "copy_bytes": 1 << 30, "source_sha256": source_sha256()}), flush=True)
        return

    if args.loop_only:
        print(json.dumps({"decode_loop": b.decode_loop()}), flush=True)
        return

    # always-Full baseline
    full = b.timed(b.full_calls(), args.warmup, cold=True)
    log(f"[bench] always-Full {full['us_mean']:.1f} us/step ({bytes_full / full['us_mean'] / 1e3:.0f} GB/s)")

    # rho sweep with the App. A.2 head (headline), then the MLP stand-in
    head0 = args.head
    sweep = run_sweep(b, wl, args, full["us_mean"])
    other = "mlp" if head0 == "paper" else "paper"
    sweep_other = []
    if not args.one_head:
        b.set_head(other)
        sweep_other = run_sweep(b, wl, args, full["us_mean"])
        b.set_head(head0)

    loop = [] if args.no_loop else b.decode_loop()
    layout = b.local_layout()
    log(f"[bench] Local alone, cold: permuted block table {layout['permuted_us']:.1f} us, "
        f"contiguous table {layout['contiguous_us']:.1f} us")

    # roofline of the dominant kernel: the Full split-K pass over every request
    # (one launch of attn_split_kernel<128, false>; no merge launch at this size),
    # the last ROOFLINE_REPS dispatches of that kernel in this process
    fcalls = b.full_calls()[0]
    t_full_call = b.kernel_time(fcalls, reps=ROOFLINE_REPS, cold=True)
    roof = dict(bound="hbm", achieved=bytes_full / t_full_call / 1e3, peak=HBM_PEAK_GBS, unit="GB/s",
                traffic=measured_traffic())
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = ROOFLINE_KERNEL + " (oda_full_decode_attn, every request)"
    roof["bytes_per_launch"] = bytes_full
    roof["us_per_launch"] = t_full_call

    head_ent = min(sweep, key=lambda e: abs(e["rho"] - HEADLINE_RHO)) if sweep else None
    value = head_ent["us"] if head_ent else full["us_mean"]
    res = {
        "metric": METRIC, "value": round(value, 3), "unit": "us/step", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(value / 1e3, 6), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.num_layers} layers, B={wl.batch}, {wl.num_q_heads}q/{wl.num_kv_heads}kv "
                               f"heads, D={wl.head_dim}, n={'/'.join(str(x) for x in sorted(set(b.seq_host.tolist()))[:4])}"
                               f"{'...' if len(set(b.seq_host.tolist())) > 4 else ''}, "
                               f"W={wl.stacks[-1].local_window}, s={wl.stacks[-1].local_sink}, paged bf16 KV "
                               f"(block 16, permuted), {args.head} recall head {wl.d_model}->{wl.d_hidden}->1, "
                               f"rho={head_ent['rho'] if head_ent else 1.0}, cold (Infinity Cache flushed between steps)",
                   "head": args.head, "seed": args.seed, "split_blocks": args.split_blocks},
        "GBps": round(head_ent["GBps"], 1) if head_ent else None,
        "always_full_us": round(full["us_mean"], 3),
        "always_full_GBps": round(bytes_full / full["us_mean"] / 1e3, 1),
        "sweep": [{k: (round(v, 4) if isinstance(v, float) else v) for k, v in e.items()} for e in sweep],
        f"sweep_{other}_head": [{k: (round(v, 4) if isinstance(v, float) else v) for k, v in e.items()}
                                for e in sweep_other],
        "decode_loop": [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in e.items()} for e in loop],
        "local_window_layout": {k: round(v, 3) for k, v in layout.items()},
        "roofline": {k: (round(v, 4) if isinstance(v, float) else v) for k, v in roof.items()},
    }
    if not args.no_cpu_baseline:
        cb = cpu_baseline(b, head_ent["rho"] if head_ent else 1.0)
        res["cpu_baseline"] = {k: (round(v, 3) if isinstance(v, float) else v) for k, v in cb.items()}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
