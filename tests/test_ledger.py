"""The bench's closed-form byte ledger agrees with the oracle's ledger (which
counts the attended positions of the access sets directly), and the closed
forms reproduce hand-computable sizes of the measured configurations."""
import numpy as np
import pytest

from oracle import ledger as OL
from paper_2609_20734_amd import ledger as PL
from paper_2609_20734_amd import workloads as WL


@pytest.mark.parametrize("n,s,w", [(1, 4, 16), (5, 4, 3), (20, 0, 5), (2052, 4, 2048), (2053, 4, 2048),
                                   (32768, 4, 1024), (33, 16, 16), (100, 40, 50), (7, 4, 0)])
def test_local_count_matches_set_size(n, s, w):
    from oracle import attention as OA
    ref = len(OA.local_set(n, s, w)) if w > 0 else n
    assert PL.local_count(n, s, w) == ref
    blocks = len(np.unique(OA.local_set(n, s, w) // 16)) if w > 0 else (n + 15) // 16
    assert PL.visited_blocks(n, s, w) == blocks


def test_attention_bytes_match_oracle_ledger():
    seq = [1, 17, 300, 2049, 5000]
    from oracle import attention as OA
    for s, w in ((4, 1024), (0, 64), (4, 0)):
        a = PL.attention_bytes(seq, s, w, 3, 16, 4, 128)
        f = (lambda n: OA.local_set(n, s, w)) if w > 0 else OA.full_set
        b = OL.attention_bytes(seq, f, 3, 16, 4, 128)
        assert a == b


def test_gate_bytes_match_oracle_ledger():
    for kind, d, dh in (("paper", 4096, 256), ("mlp", 4096, 256), ("paper", 8192, 512)):
        assert PL.gate_bytes(kind, 8, d, dh) == OL.gate_bytes(kind, 8, d, dh)
    assert PL.gate_param_count("paper", 2048, 1024) == 28_325_889


def test_llama_config_sizes():
    wl = WL.LLAMA
    full = PL.attention_bytes(wl.seq_lens, 0, 0, 32, 32, 8, 128)
    assert full["kv"] == 32 * 8 * 32768 * 4 * 128 == 4_294_967_296
    loc = PL.attention_bytes(wl.seq_lens, 4, 1024, 32, 32, 8, 128)
    assert loc["kv"] == 32 * 8 * 1028 * 512


def _kv(wl, seq, stacks, local):
    tot = 0
    for st in stacks:
        if local:
            s, w = (st.local_sink, st.local_window) if st.gated else (0, st.native_window)
        else:
            s, w = 0, st.native_window
        tot += PL.attention_bytes(seq, s, w, st.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim)["kv"]
    return tot


@pytest.mark.parametrize("name,rhos,want,gated_only", [
    ("llama3-8b", (0, .1, .25, .5, 1), (0.032, 0.132, 0.282, 0.532, 1.032), False),
    ("long", (0, .05, .2, 1), (0.031, 0.081, 0.231, 1.031), False),
    ("hybrid", (0, .1, .25, .5, 1), (0.211, 0.311, 0.461, 0.711, 1.211), False),
    ("hybrid", (0, .1, .25, .5, 1), (0.211, 0.295, 0.422, 0.632, 1.053), True)])
def test_ideal_ratios_match_independent_ledger(name, rhos, want, gated_only):
    """Ideal bytes ratios (KV + MLP-head weights) of the measured
    configurations, computed independently from the configuration sizes:
    Bytes(rho) / Bytes_Full with the retry over every layer, or over the gated
    layers only.  The bench's own ratio (which also counts q, out, lse and
    block tables) stays within 0.001 of them."""
    import bench as BN
    wl = WL.ALL[name]
    seq = np.array(wl.seq_lens)
    full = _kv(wl, seq, wl.stacks, False)
    local = _kv(wl, seq, wl.stacks, True)
    retry = _kv(wl, seq, [st for st in wl.stacks if st.gated or not gated_only], False)
    gate = PL.gate_bytes("mlp", wl.batch, wl.d_model, wl.d_hidden)["weights"]
    for rho, w in zip(rhos, want):
        assert round((local + gate + rho * retry) / full, 3) == w
        lb, gb, fb = BN.bytes_for(wl, seq, None, "mlp", gated_only)
        _, _, fall = BN.bytes_for(wl, seq, None, "mlp")
        bench_ratio = (lb + gb + rho * sum(fb)) / sum(fall)
        assert abs(bench_ratio - (local + gate + rho * retry) / full) < 1e-3


def test_always_full_bytes_of_the_llama_stack_by_hand():
    """Bytes_Full of one 32-layer step over 32,768 positions, added up by hand:
    K + V rows 32 layers x 8 KV heads x 32,768 positions x 512 B = 4,294,967,296;
    q 32 x 32 heads x 128 x 2 B = 262,144; out + lse 32 x 32 x 129 x 4 B = 528,384;
    2,048 block-table entries x 4 B = 8,192."""
    got = OL.always_full_bytes([32768], 0, 32, 32, 8, 128)
    assert got == 4_294_967_296 + 262_144 + 528_384 + 8_192 == 4_295_766_016


def test_step_bytes_by_hand_and_limits():
    """Bytes(rho) of a small step, by hand: two requests of 40 and 9 positions,
    one layer, 2 query / 1 KV head of 16 (64 B per position), s = 4, w = 8,
    the MLP head 8 -> 4 -> 1.
      Local: request 0 attends 4 + 8 = 12 positions in blocks {0, 2} -> 768 B
             of K/V + 2 table entries; request 1 (n = 9) attends all 9 -> 576 B
             + 1 entry; q 2 x 64 B, out + lse 2 x 2 x 17 x 4 B.
      Gate: (4 x 8 + 4 + 4 + 1) x 4 B weights + 2 x 8 x 4 B inputs + 2 x 12 + 12 B.
      Full (request 0 flagged): 40 x 64 B + 3 entries + 64 B q + 136 B out."""
    seq = [40, 9]
    local = (12 * 64 + 2 * 4) + (9 * 64 + 1 * 4) + 2 * 64 + 2 * 136
    gate = (4 * 8 + 4 + 4 + 1) * 4 + 2 * 8 * 4 + 2 * 12 + 12
    full = 40 * 64 + 3 * 4 + 64 + 136
    got = OL.step_bytes(seq, [1, 0], 4, 8, 0, 1, 2, 1, 16, "mlp", 8, 4)
    assert got == dict(local=local, gate=gate, full=full, total=local + gate + full)
    none = OL.step_bytes(seq, [0, 0], 4, 8, 0, 1, 2, 1, 16, "mlp", 8, 4)
    assert none["full"] == 0 and none["total"] == local + gate
    # a window that covers every history: Local reads exactly what Full reads
    cover = OL.step_bytes(seq, [1, 1], 4, 64, 0, 1, 2, 1, 16, "mlp", 8, 4)
    assert cover["local"] == cover["full"] == OL.always_full_bytes(seq, 0, 1, 2, 1, 16)


def test_gate_bytes_of_the_paper_head_at_qwen3_width():
    """App. A.2's head for d = 2048 has 28,325,889 fp32 parameters."""
    g = OL.gate_bytes("paper", 1, 2048, 1024)
    assert g["weights"] == 4 * 28_325_889
    assert g["inputs"] == 3 * 2048 * 4
