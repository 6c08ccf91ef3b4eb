"""Host-side logic of bench.py, on the CPU: the one-GPU guard, the keyed
HBM-traffic lookup, threshold calibration, and the flag comparison with the
oracle's decisions (borderline counting)."""
import json
import math
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench as BN  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_taus_flag_the_requested_number_of_decisions():
    scores = np.random.default_rng(1).standard_normal((50, 32))
    taus = BN.taus_for(scores, (0.0, 0.1, 0.25, 1.0))
    assert taus[0.0] == math.inf and taus[1.0] == -math.inf
    for rho in (0.1, 0.25):
        # round(rho N) flagged, give or take the few decisions a narrow gap moves it by
        assert abs(int((scores > taus[rho]).sum()) - round(rho * scores.size)) <= 3
        assert np.abs(scores - taus[rho]).min() >= BN.FLAG_BORDER   # no borderline decision at the threshold


def test_taus_avoid_narrow_gaps():
    """A gap below 2e-4 between the scores around the quantile moves the
    threshold to the nearest wide gap, so no decision at it is borderline."""
    s = np.array([5.0, 4.0, 3.0, 2.00005, 2.0, 1.0, 0.0, -1.0, -2.0, -3.0])
    tau = BN.taus_for(s, (0.4,))[0.4]          # 4 of 10: the gap 2.00005 | 2.0 is too narrow
    assert tau == 0.5 * (3.0 + 2.00005)          # the nearest wide gap (one fewer flagged)
    assert np.abs(s - tau).min() >= 1e-4
    tau = BN.taus_for(s, (0.5,))[0.5]          # 5 of 10: the gap 2.0 | 1.0 is wide already
    assert tau == 1.5
    tau = BN.taus_for(s, (0.3,))[0.3]          # 3 of 10: gap 3.0 | 2.00005 is wide
    assert tau == 0.5 * (3.0 + 2.00005)


def test_flags_vs_oracle_counts_borderline_and_mismatches():
    score = np.array([[0.5, 0.00005, -0.2, np.nan], [0.3, -0.00005, 0.1, np.inf]])
    tau = 0.0
    want = np.array([[1, 1, 0, 1], [1, 0, 1, 1]], dtype=np.int32)   # strict >, nonfinite -> Full
    # kernel agrees everywhere except one borderline decision and one clear one
    gpu = want.copy()
    gpu[0, 1] = 0            # |score - tau| = 5e-5 < 1e-4: borderline, decided differently
    gpu[1, 2] = 0            # a clear mismatch
    r = BN.flags_vs_oracle(gpu, score, tau, None)
    assert r == dict(decisions=8, borderline=2, flag_mismatch=1, borderline_differ=1)
    # prescribed flags: no borderline band; nonfinite scores still go to Full
    forced = np.array([[0, 1, 0, 0], [1, 0, 0, 0]], dtype=np.int32)
    expect = np.array([[0, 1, 0, 1], [1, 0, 0, 1]], dtype=np.int32)
    r = BN.flags_vs_oracle(expect, score, tau, forced)
    assert r == dict(decisions=8, borderline=0, flag_mismatch=0, borderline_differ=0)


@pytest.fixture
def traffic_dir(tmp_path, monkeypatch):
    """bench.py reading its counter summary from a scratch copy of the tree."""
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(BN, "ROOT", str(tmp_path))
    return tmp_path


def _write_summary(d, workload, nbytes, sha, traffic=123456):
    (d / "profiles" / f"full_split_{workload}_traffic.txt").write_text(
        "# header\n"
        f"workload_name: {workload}\n"
        f"algorithmic_bytes_per_launch: {nbytes}\n"
        f"traffic_bytes_per_launch: {traffic}\n"
        f"source_sha256: {sha}\n")


def test_traffic_is_reported_only_for_the_matching_workload_size_and_source(traffic_dir):
    sha = BN.source_sha256()
    assert BN.measured_traffic("mixed", 1000) is None                     # no summary
    _write_summary(traffic_dir, "mixed", 1000, sha)
    assert BN.measured_traffic("mixed", 1000) == 123456.0
    assert BN.measured_traffic("mixed", 1001) is None                     # another launch size
    assert BN.measured_traffic("long", 1000) is None                      # another workload's file is absent
    _write_summary(traffic_dir, "mixed", 1000, "0" * 64)
    assert BN.measured_traffic("mixed", 1000) is None                     # kernel source changed
    _write_summary(traffic_dir, "long", 1000, sha)
    (traffic_dir / "profiles" / "full_split_long_traffic.txt").write_text(
        (traffic_dir / "profiles" / "full_split_long_traffic.txt").read_text().replace("workload_name: long",
                                                                                      "workload_name: mixed"))
    assert BN.measured_traffic("long", 1000) is None                      # a file naming another workload


def test_committed_summaries_match_their_workloads():
    """Every committed counter summary names its own workload and a launch size
    the ledger reproduces; the default workload's summary carries the current
    kernel source's hash (so the default bench line reports traffic)."""
    from paper_2609_20734_amd import workloads as WL
    for name in ("mixed", "llama3-8b"):
        path = os.path.join(ROOT, "profiles", f"full_split_{name}_traffic.txt")
        vals = dict(l.split(":", 1) for l in open(path) if ":" in l and not l.startswith("#"))
        vals = {k.strip(): v.strip() for k, v in vals.items()}
        assert vals["workload_name"] == name
        wl = WL.ALL[name]
        seq = BN.workload_seq_lens(wl, 1234)
        _, _, full_b = BN.bytes_for(wl, seq, None, "paper")
        assert int(vals["algorithmic_bytes_per_launch"]) == sum(full_b)
        assert 1.0 <= float(vals["traffic_over_algorithmic"]) < 1.01
    mixed = open(os.path.join(ROOT, "profiles", "full_split_mixed_traffic.txt")).read()
    assert f"source_sha256: {BN.source_sha256()}" in mixed
