"""bench.py's output on the smallest workload (one layer, 1 x 1,024 positions,
W = 128), run as a process of its own: one JSON line on stdout with the
fields a driver reads, a roofline object that recomputes from its own
figures, the CPU oracle leg, and every timed operating point's flags equal
to the fp64 oracle head's (borderline decisions aside)."""
import json
import math
import os
import subprocess
import sys

import pytest

from harness import need_gpu

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
STEPS, WARMUP = 8, 2


@pytest.fixture(scope="module")
def line():
    need_gpu()
    print("[bench contract] bench.py --config tiny", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--config", "tiny",
                        "--steps", str(STEPS), "--warmup", str(WARMUP), "--reps", "1", "--extra-configs", ""],
                       cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, lines[:3]          # the one JSON line; progress goes to stderr
    return json.loads(lines[0])


def test_driver_fields(line):
    sys.path.insert(0, ROOT)
    import bench as BN
    d = line
    assert d["metric"] == BN.METRIC and d["unit"] == "us/step"
    assert d["n_gpus"] == 1 and d["steps"] == STEPS and d["warmup"] == WARMUP
    assert d["value"] > 0 and math.isclose(d["ms_per_step"], d["value"] / 1e3, rel_tol=1e-4)
    assert d["higher_is_better"] is False and d["scaling"] == "weak" and d["vs_baseline"] is None
    assert d["dtype"] == "bf16" and d["data"] == "synthetic"
    assert d["config"]["workload"].startswith("tiny:")
    assert not any(k in d["config"] for k in ("model", "global_batch", "seq_len"))


def test_roofline_recomputes(line):
    roof = line["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert math.isclose(roof["achieved"], roof["bytes_per_launch"] / roof["us_per_launch"] / 1e3, rel_tol=1e-3)
    assert math.isclose(roof["frac"], roof["achieved"] / roof["peak"], abs_tol=1e-4)   # printed to 4 places
    assert roof["traffic"] is None        # no counter summary is kept for this workload
    assert 0 < roof["frac"] < 1


def test_cpu_leg_and_oracle_flags(line):
    cb = line["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    assert cb["pool"]["kind"] == "oracle" and cb["pool"]["cores"] >= 1
    assert line["sweep"]
    for pt in line["sweep"]:
        f = pt["flags_vs_oracle"]
        assert f["decisions"] == STEPS * 1          # batch 1, every timed step
        assert f["flag_mismatch"] == 0, pt
        # the threshold sits in a score gap at least twice the borderline band wide
        assert f["borderline"] == 0, pt
