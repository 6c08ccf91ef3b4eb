"""Synthetic decode workloads shaped like the paper's long-context decoding
(§3, App. B.7: bf16 KV, GQA, sinks s = 4, long histories) at the sizes of
the five measured configurations.  Shapes only; values come from oda_synth.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Stack:
    """One group of layers sharing the same access-set parameters."""
    name: str
    num_layers: int
    local_sink: int       # Local sinks s (ignored when local_window == native_window and native)
    local_window: int     # Local window w (current token included)
    native_window: int    # 0: full-history layer; > 0: natively sliding-window layer
    gated: bool           # restricted by ODA (True) or native in both branches (False)


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    stacks: tuple
    seq_lens: tuple = ()              # fixed lengths (one per request), or
    seq_range: tuple = ()             # (lo, hi): seeded uniform lengths
    permute: bool = True
    d_model: int = 0
    d_hidden: int = 0
    rhos: tuple = ()                  # recall rates swept via the threshold
    bernoulli: tuple = ()             # per-request forced-flag probabilities (when set, the headline
                                      # operating points; threshold-driven rates are reported beside them)
    steps: int = 16
    extra: dict = field(default_factory=dict)

    @property
    def num_layers(self) -> int:
        return sum(s.num_layers for s in self.stacks)


def _gated(L, W, s=4):
    return Stack("global", L, s, W, 0, True)


TINY = Workload("tiny", batch=1, num_q_heads=8, num_kv_heads=2, head_dim=64, stacks=(_gated(1, 128),),
                seq_lens=(1024,), permute=False, d_model=512, d_hidden=64, rhos=(5 / 16,), steps=16)

LLAMA = Workload("llama3-8b", batch=1, num_q_heads=32, num_kv_heads=8, head_dim=128, stacks=(_gated(32, 1024),),
                 seq_lens=(32768,), d_model=4096, d_hidden=256, rhos=(0.0, 0.1, 0.25, 0.5, 1.0), steps=1000)

MIXED = Workload("mixed", batch=32, num_q_heads=32, num_kv_heads=8, head_dim=128, stacks=(_gated(32, 2048),),
                 seq_range=(8192, 65536), d_model=4096, d_hidden=256, rhos=(0.1, 0.25, 0.5),
                 bernoulli=(0.0, 0.1, 0.25, 0.5), steps=50)

LONG = Workload("long", batch=4, num_q_heads=32, num_kv_heads=8, head_dim=128, stacks=(_gated(32, 4096),),
                seq_lens=(131072,) * 4, d_model=4096, d_hidden=256, rhos=(0.0, 0.05, 0.2, 1.0), steps=100)

HYBRID = Workload("hybrid", batch=8, num_q_heads=64, num_kv_heads=8, head_dim=128,
                  stacks=(Stack("swa", 36, 0, 4096, 4096, False), Stack("global", 12, 4, 4096, 0, True)),
                  seq_lens=(65536,) * 8, d_model=8192, d_hidden=512, rhos=(0.0, 0.1, 0.25, 0.5, 1.0), steps=100)

ALL = {w.name: w for w in (TINY, LLAMA, MIXED, LONG, HYBRID)}
