"""Host-side parts of bench.py that run without a GPU: the CPU-baseline leg
(the oracle on a bounded sample), the one-GPU guard, and the summaries of
rocprofv3 kernel traces and HBM counters behind the committed profiles."""
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


def _write_csv(path, header, rows):
    import csv
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_summarize_trace_tables(tmp_path):
    # per-kernel totals over every launch; the copy kernels' full-slot table
    # keeps only the launches of the largest grid
    import bench
    pack, unpack = list(bench.PMC_KERNELS)
    rows = [  # name, start ns, end ns, grid x
        (pack, 0, 300_000, 2_097_152), (pack, 0, 360_000, 2_097_152), (pack, 0, 10_000, 4_096),
        (unpack, 0, 380_000, 2_097_152), (unpack, 0, 5_000, 8_192),
        ("void ss::k_plan_core(ss::PlanArgs)", 0, 40_000, 1_024),
    ]
    csv_path = tmp_path / "run_kernel_trace.csv"
    _write_csv(csv_path, ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"], rows)
    md = bench.summarize_trace(str(csv_path), str(tmp_path / "out.md"), "T", "cmd")
    assert "| `ss::k_copy<true>` | 3 | 0.67 | 223.3 | 10.0 | 360.0 |" in md
    assert "| `ss::k_copy<false>` | 2 | 0.39 | 192.5 | 5.0 | 380.0 |" in md
    assert "| `ss::k_plan_core` | 1 | 0.04 | 40.0 | 40.0 | 40.0 |" in md
    assert "| `pack` | 2,097,152 | 2 | 330.0 | 330.0 | 300.0 |" in md
    assert "| `unpack` | 2,097,152 | 1 | 380.0 | 380.0 | 380.0 |" in md


def test_summarize_pmc_scales_by_the_probe(tmp_path):
    # The probe's plain copy reads and writes PROBE_BYTES; counters that read
    # half (FETCH) and exactly (WRITE) that on it give scale factors 2 and 1.
    # Copy kernels over a whole 1 GiB slot of the round-robin layout (512
    # units of 2 MiB; pack grid 512 x 8 blocks, unpack 64 x 64 blocks) whose
    # scaled counters equal one read and one write of the slot have a traffic
    # ratio of exactly 1.
    import bench
    pack, unpack = list(bench.PMC_KERNELS)
    kib = bench.PROBE_BYTES / 1024
    slot_kib = 512 * (2 << 20) / 1024
    grid = 4096 * bench.COPY_BLOCK
    fetch = [(bench.PROBE_KERNEL, "FETCH_SIZE", kib / 2, 1 << 20),
             (pack, "FETCH_SIZE", slot_kib / 2, grid), (pack, "FETCH_SIZE", 1.0, 1024),
             (unpack, "FETCH_SIZE", slot_kib / 2, grid)]
    write = [(bench.PROBE_KERNEL, "WRITE_SIZE", kib, 1 << 20),
             (pack, "WRITE_SIZE", slot_kib, grid), (pack, "WRITE_SIZE", 1.0, 1024),
             (unpack, "WRITE_SIZE", slot_kib, grid)]
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value", "Grid_Size"]
    _write_csv(tmp_path / "f.csv", hdr, fetch)
    _write_csv(tmp_path / "w.csv", hdr, write)
    out = bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "roundrobin",
                              str(tmp_path / "pmc.json"), ["cmd"])
    assert abs(out["probe_scale_factor"]["FETCH_SIZE"] - 2.0) < 1e-12
    assert abs(out["probe_scale_factor"]["WRITE_SIZE"] - 1.0) < 1e-12
    for short in ("pack", "unpack"):
        k = out["kernels"][short]
        assert k["units_per_launch"] == 512 and k["dispatches"] == 1
        assert abs(k["traffic_over_algorithmic"] - 1.0) < 1e-12
    assert out["kernel_source_sha256_16"] == bench.kernel_source_hash()
