"""Host-side parts of bench.py that run without a GPU: the CPU-baseline leg
(the oracle on a bounded sample) and the one-GPU guard."""
import subprocess
import sys
import os

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_baseline_leg_runs_on_a_sample():
    import bench
    tr = W.make_trace("tiny", 0)
    rec = bench.cpu_baseline(tr, 5, 3, 4, W.SENTINEL, None)
    assert rec["kind"] == "oracle" and rec["cores"] == 1 and rec["unit"] == "GB/s"
    assert rec["value"] > 0
    assert "steps 5-7 of the tiny trace" in rec["sample"]


def test_cpu_baseline_leg_with_a_budget_and_threshold():
    import bench
    tr = W.make_trace("tiny", 1)
    rec = bench.cpu_baseline(tr, 10, 2, 2, 3, 8)
    assert rec["value"] > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
