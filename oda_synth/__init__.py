"""Seeded synthetic inputs for the ODA decode-step hot path.

This module is shared by the fp64 oracle side (tests, the CPU baseline) and
the HIP side (tests, bench).  It holds no arithmetic of the method itself:
it only draws numbers, rounds them to the storage formats the C ABI takes,
and lays them out in the ABI's memory layouts.

Value distributions follow the workloads the paper times (long-context
decoding, bf16 KV, GQA; §3 and App. B.7) with i.i.d. N(0,1) activations as a
stand-in for real prompts:

* q, K, V: N(0,1) rounded to bf16 (round to nearest even);
* gate inputs (h_prev, E(x_t), h^L): N(0,1) in fp32;
* gate weights and biases 0.02*N(0,1); RMSNorm gains 1 + 0.02*N(0,1);
* block tables: a seeded permutation of all physical blocks.

Host generation uses numpy's PCG64 seeded by (seed, stream id).  Large
device-resident caches are filled on the GPU with torch's Philox generator
(``fill_normal_bf16_``); the oracle then reads back only the slices it
checks, so every oracle input is a copy of what the kernels read.
"""
from __future__ import annotations

import numpy as np

BLOCK_SIZE = 16

# Stream ids: one per tensor so that changing one shape never changes the
# values of another tensor.
STREAM_Q = 1
STREAM_K = 2
STREAM_V = 3
STREAM_TABLE = 4
STREAM_KCUR = 5
STREAM_VCUR = 6
STREAM_GATE_PARAMS = 7
STREAM_GATE_INPUTS = 8
STREAM_SEQ_LENS = 9
STREAM_FORCED = 10
STREAM_DECODER = 11
STREAM_TOKENS = 12


def rng(seed: int, stream: int) -> np.random.Generator:
    """Independent PCG64 stream for (seed, stream)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(stream)])))


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return raw uint16 bits."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint32)
    nan = np.isnan(x)
    r = np.where(nan, (u >> 16).astype(np.uint32) | 0x40, r)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    """Exact widening of raw bf16 bits to float32 (for building inputs only)."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16)).astype(np.uint32) << 16
    return b.view(np.float32)


def normal_bf16(g: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    """N(0, std^2) samples rounded to bf16, as raw uint16 bits."""
    x = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x = (x * np.float32(std)).astype(np.float32)
    return f32_to_bf16_bits(x)


def paged_block_table(g: np.random.Generator, seq_lens, max_blocks_per_seq: int | None = None,
                      permute: bool = True, extra_blocks: int = 0):
    """Assign physical KV blocks to every request.

    Request b owns ceil(n_b/16) logical blocks.  With ``permute`` the physical
    ids are a seeded permutation of all blocks (shared by every layer); without
    it they are contiguous (identity layout).  Unused table entries are 0.
    Returns (block_table int32 [B][max_blocks_per_seq], num_blocks).
    """
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    need = (seq_lens + BLOCK_SIZE - 1) // BLOCK_SIZE
    if max_blocks_per_seq is None:
        max_blocks_per_seq = int(need.max()) if len(need) else 1
    total = int(need.sum()) + int(extra_blocks)
    ids = g.permutation(total) if permute else np.arange(total)
    table = np.zeros((len(seq_lens), max_blocks_per_seq), dtype=np.int32)
    pos = 0
    for b, nb in enumerate(need):
        table[b, :nb] = ids[pos:pos + nb]
        pos += int(nb)
    return table, max(total, 1)


def kv_cache_shapes(num_layers: int, num_blocks: int, num_kv_heads: int, head_dim: int):
    """ABI layouts of the paged caches (element = one bf16).

    K: [L][num_blocks][Hkv][D/8][16][8] -- 16-byte groups of 8 dims, token-minor.
    V: [L][num_blocks][Hkv][D][16]      -- dims-major, the 16 tokens of a block contiguous.
    """
    k = (num_layers, num_blocks, num_kv_heads, head_dim // 8, BLOCK_SIZE, 8)
    v = (num_layers, num_blocks, num_kv_heads, head_dim, BLOCK_SIZE)
    return k, v


def kv_cache(seed: int, num_layers: int, num_blocks: int, num_kv_heads: int, head_dim: int):
    """Host-generated K and V caches (uint16 bf16 bits) in the ABI layouts."""
    ks, vs = kv_cache_shapes(num_layers, num_blocks, num_kv_heads, head_dim)
    return normal_bf16(rng(seed, STREAM_K), ks), normal_bf16(rng(seed, STREAM_V), vs)


# --------------------------------------------------------------------------
# recall-gate parameters (packed fp32, ABI order)
# --------------------------------------------------------------------------

def paper_head_segments(d: int, dt: int):
    """(name, kind, count) in the packed order the ABI defines for the
    App. A.2 head; kind is 'w' (weight/bias) or 'g' (RMSNorm gain)."""
    segs = []
    for t in ("h", "e", "l"):
        segs += [(f"rms_{t}", "g", d), (f"W_{t}", "w", dt * d), (f"b_{t}", "w", dt)]
    segs += [("W_f", "w", dt * 9 * dt), ("b_f", "w", dt)]
    for k in (1, 2):
        segs += [(f"rms_{k}", "g", dt), (f"W_gate_{k}", "w", 2 * dt * dt),
                 (f"W_up_{k}", "w", 2 * dt * dt), (f"W_down_{k}", "w", dt * 2 * dt)]
    segs += [("rms_o", "g", dt), ("w_o", "w", dt), ("b_o", "w", 1)]
    return segs


def mlp_segments(d: int, h: int):
    return [("W1", "w", h * d), ("b1", "w", h), ("w2", "w", h), ("b2", "w", 1)]


def gate_params(seed: int, kind: str, d: int, dh: int) -> np.ndarray:
    """Packed fp32 gate parameters: weights/biases 0.02*N(0,1), gains 1+0.02*N(0,1)."""
    segs = paper_head_segments(d, dh) if kind == "paper" else mlp_segments(d, dh)
    g = rng(seed, STREAM_GATE_PARAMS)
    out = []
    for _, k, cnt in segs:
        x = (0.02 * g.standard_normal(cnt)).astype(np.float32)
        if k == "g":
            x = (1.0 + x.astype(np.float64)).astype(np.float32)
        out.append(x)
    return np.concatenate(out).astype(np.float32)


def gate_inputs(seed: int, steps: int, batch: int, d: int, stream_offset: int = 0):
    """fp32 N(0,1) gate inputs h_prev, E(x_t), h^L, each [steps][B][d]."""
    g = rng(seed + stream_offset, STREAM_GATE_INPUTS)
    x = g.standard_normal((3, steps, batch, d), dtype=np.float32)
    return x[0], x[1], x[2]


def uniform_seq_lens(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """Per-request context lengths, uniform integers in [lo, hi]."""
    return rng(seed, STREAM_SEQ_LENS).integers(lo, hi + 1, size=batch).astype(np.int32)


def bernoulli_flags(seed: int, steps: int, batch: int, p: float) -> np.ndarray:
    """Prescribed per-request Full flags ~ Bernoulli(p), int32 [steps][B]."""
    return (rng(seed, STREAM_FORCED).random((steps, batch)) < p).astype(np.int32)


def periodic_schedule(steps: int, first_k: int, period: int = 16) -> np.ndarray:
    """Device-side schedule of the runtime protocol: Full for the first
    ``first_k`` steps of every ``period``-step period (App. B.7)."""
    return (np.arange(steps) % period < first_k).astype(np.int32)


# --------------------------------------------------------------------------
# device fill for caches too large to build on the host
# --------------------------------------------------------------------------

def fill_normal_bf16_(t, seed: int, stream: int, chunk_elems: int = 1 << 28, std: float = 1.0) -> None:
    """Fill a CUDA tensor (dtype bfloat16 or int16 view of one) with N(0, std^2)
    bf16 values drawn from torch's Philox generator, in chunks."""
    import torch
    g = torch.Generator(device=t.device)
    g.manual_seed(int(seed) * 1000003 + int(stream))
    flat = t.view(-1)
    if flat.dtype != torch.bfloat16:
        flat = flat.view(torch.bfloat16)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        flat[s:e].normal_(0.0, float(std), generator=g)


# ---------------------------------------------------------------------------
# the decoder around the hot path (synthetic weights of a given shape)
# ---------------------------------------------------------------------------

def decoder_tensor_specs(L: int, d: int, Hq: int, Hkv: int, D: int, F: int, V: int):
    """(name, shape, kind, std) of every decoder tensor.  kind "w": bf16 weight
    ~ N(0, std^2); "g": fp32 RMSNorm gain 1 + 0.02 N(0,1).  Dense weights are
    [out][in]; w_gu holds the F gate rows then the F up rows; the vocabulary
    projection is the embedding table (tied)."""
    qkv = (Hq + 2 * Hkv) * D
    return [("embed", (V, d), "w", 1.0),
            ("attn_norm", (L, d), "g", 0.0),
            ("w_qkv", (L, qkv, d), "w", d ** -0.5),
            ("q_norm", (L, D), "g", 0.0),
            ("k_norm", (L, D), "g", 0.0),
            ("w_o", (L, d, Hq * D), "w", (Hq * D) ** -0.5),
            ("mlp_norm", (L, d), "g", 0.0),
            ("w_gu", (L, 2 * F, d), "w", d ** -0.5),
            ("w_down", (L, d, F), "w", F ** -0.5),
            ("final_norm", (d,), "g", 0.0)]


def decoder_weights(seed: int, L: int, d: int, Hq: int, Hkv: int, D: int, F: int, V: int) -> dict:
    """Host arrays (bf16 bits as uint16, gains as float32) for small shapes."""
    g = rng(seed, STREAM_DECODER)
    out = {}
    for name, shape, kind, std in decoder_tensor_specs(L, d, Hq, Hkv, D, F, V):
        if kind == "w":
            out[name] = normal_bf16(g, shape, std)
        else:
            out[name] = (1.0 + 0.02 * g.standard_normal(shape)).astype(np.float32)
    return out


def decoder_weights_device(seed: int, L: int, d: int, Hq: int, Hkv: int, D: int, F: int, V: int, device) -> dict:
    """Device tensors of the same tensors, filled with torch's Philox generator
    (full-size models; not the same values as decoder_weights)."""
    import torch
    out = {}
    for i, (name, shape, kind, std) in enumerate(decoder_tensor_specs(L, d, Hq, Hkv, D, F, V)):
        if kind == "w":
            t = torch.empty(shape, dtype=torch.bfloat16, device=device)
            fill_normal_bf16_(t, seed, STREAM_DECODER * 100 + i, std=std)
        else:
            t = torch.empty(shape, dtype=torch.float32, device=device)
            gen = torch.Generator(device=device)
            gen.manual_seed(int(seed) * 1000003 + STREAM_DECODER * 100 + i)
            t.normal_(0.0, 0.02, generator=gen).add_(1.0)
        out[name] = t
    return out


def tokens(seed: int, steps: int, batch: int, vocab: int) -> np.ndarray:
    """A fixed continuation: uniform token ids, int32 [steps][B]."""
    return rng(seed, STREAM_TOKENS).integers(0, vocab, size=(steps, batch)).astype(np.int32)
