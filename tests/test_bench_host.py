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


def test_launch_units_by_layout():
    # pack: ceil(items / 8) workgroups per unit.  Unpack with one item per
    # plane (64 x 32 KiB KV pages) runs n_items workgroups per 8 units; with
    # several items per plane (one 512 KiB plane = 16 items) it takes the pack
    # order.
    import bench
    assert bench.launch_units("pack", 4096, 64, 64) == 512
    assert bench.launch_units("unpack", 4096, 64, 64) == 512
    assert bench.launch_units("pack", 4096, 16, 1) == 2048
    assert bench.launch_units("unpack", 4096, 16, 1) == 2048


def test_summarize_pmc_diffusion_layout(tmp_path):
    # a whole 1 GiB slot of the diffusion layout is 2,048 units of 512 KiB:
    # 4,096 workgroups for the pack and (pack order) for the unpack
    import bench
    pack, unpack = list(bench.PMC_KERNELS)
    kib = bench.PROBE_BYTES / 1024
    slot_kib = 2048 * (512 << 10) / 1024
    grid = 4096 * bench.COPY_BLOCK
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value", "Grid_Size"]
    _write_csv(tmp_path / "f.csv", hdr, [(bench.PROBE_KERNEL, "FETCH_SIZE", kib / 2, 1 << 20),
                                         (pack, "FETCH_SIZE", slot_kib / 2, grid),
                                         (unpack, "FETCH_SIZE", 1.01 * slot_kib / 2, grid)])
    _write_csv(tmp_path / "w.csv", hdr, [(bench.PROBE_KERNEL, "WRITE_SIZE", kib, 1 << 20),
                                         (pack, "WRITE_SIZE", slot_kib, grid),
                                         (unpack, "WRITE_SIZE", 1.01 * slot_kib, grid)])
    out = bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "diffusion",
                              str(tmp_path / "pmc.json"), ["cmd"])
    assert out["kernels"]["pack"]["units_per_launch"] == 2048
    assert out["kernels"]["unpack"]["units_per_launch"] == 2048
    assert abs(out["kernels"]["pack"]["traffic_over_algorithmic"] - 1.0) < 1e-12
    assert abs(out["kernels"]["unpack"]["traffic_over_algorithmic"] - 1.01) < 1e-12


def test_summarize_trace_all_launch_rate(tmp_path):
    # two whole-slot packs of the diffusion layout (2 GiB algorithmic bytes
    # each) in 250 + 286.9 us, and a half-slot one in 250 us: 5 GiB / 786.9 us
    import bench
    pack, _ = list(bench.PMC_KERNELS)
    rows = [(pack, 0, 250_000, 4096 * 512), (pack, 0, 286_900, 4096 * 512),
            (pack, 0, 250_000, 2048 * 512)]
    csv_path = tmp_path / "run_kernel_trace.csv"
    _write_csv(csv_path, ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"], rows)
    md = bench.summarize_trace(str(csv_path), str(tmp_path / "out.md"), "T", "cmd",
                               workload="diffusion")
    tbs = 5 * (1 << 30) / 786.9e-6 / 1e12
    assert f"| `pack` | 3 | {5 * (1 << 30) / 1e9:.1f} | 787 | {tbs:.2f} | {tbs / 8:.3f} |" in md


def test_summarize_copies(tmp_path):
    # device-to-host copies on two streams (the probe's one copy, the step
    # stream's three), host-to-device on one; busy time is the union of each
    # stream's intervals, bytes come from the step records
    import json
    import bench
    hdr = ["Kind", "Direction", "Stream_Id", "Source_Agent_Id", "Destination_Agent_Id",
           "Correlation_Id", "Start_Timestamp", "End_Timestamp"]
    D, H = "MEMORY_COPY_DEVICE_TO_HOST", "MEMORY_COPY_HOST_TO_DEVICE"
    rows = [("MEMORY_COPY", D, 9, "a", "b", 1, 0, 50_000_000),                 # probe
            ("MEMORY_COPY", D, 3, "a", "b", 2, 100_000_000, 110_000_000),
            ("MEMORY_COPY", D, 3, "a", "b", 3, 105_000_000, 120_000_000),     # overlaps
            ("MEMORY_COPY", D, 3, "a", "b", 4, 120_500_000, 130_500_000),
            ("MEMORY_COPY", H, 4, "a", "b", 5, 100_000_000, 125_000_000)]
    _write_csv(tmp_path / "mc.csv", hdr, rows)
    with open(tmp_path / "steps.jsonl", "w") as f:
        f.write(json.dumps({"t": 0, "bytes_out": 1_000_000_000, "bytes_in": 2_000_000_000}) + "\n")
        f.write(json.dumps({"t": 1, "bytes_out": 500_000_000, "bytes_in": 0,
                            "direct_out_bytes": 0}) + "\n")
    with open(tmp_path / "bench.json", "w") as f:
        f.write(json.dumps({"value": 90.0, "probe": {"d2h_GBps": 60.0, "h2d_GBps": 100.0,
                                                    "duplex_GBps": 120.0},
                            "dma": {"frac_of_measured_link": 0.9}}) + "\n")
    md = bench.summarize_copies(str(tmp_path / "mc.csv"), str(tmp_path / "steps.jsonl"),
                                str(tmp_path / "bench.json"), str(tmp_path / "o.md"), "T", "cmd")
    # D2H: 1.5 GB over 30 ms busy = 50 GB/s, 0.833 of 60; H2D: 2 GB over 25 ms = 80 GB/s
    # median idle gap between successive step copies: the second overlaps the
    # first (skipped), the third starts 0.5 ms after the second ends; H2D has
    # one copy (no gap)
    assert "| device to host | 3 | 11666.7 | 500.0 | 30.0 | 1.50 | 50.0 | 60.0 | 0.833 |" in md
    assert "| host to device | 1 | 25000.0 | nan | 25.0 | 2.00 | 80.0 | 100.0 | 0.800 |" in md
    # both: 3.5 GB over the union [100, 130.5] = 30.5 ms = 114.8 GB/s
    assert "3.50 GB over 30.5 ms" in md and "= 114.8 GB/s" in md and "(0.956)" in md


def test_whole_slot_grids_by_layout():
    # 1 GiB slots (8 GiB of staging, four slots per direction): 512 round-robin
    # units (pack 8 workgroups per unit, unpack 64 workgroups per 8 units),
    # 2,048 diffusion units (2 workgroups per unit both ways) and 12 LoRA
    # adapter slots of 80 MiB (2,560 items: 320 workgroups per unit both ways)
    import bench
    import workloads as W
    kv, lora = W.make_trace("zipf_lora", 0).pools
    rr = W.make_trace("roundrobin", 0).pools[0]
    for kind in ("pack", "unpack"):
        assert bench.whole_slot_grid(kind, rr, 8192 << 20, 4) == 4096 * bench.COPY_BLOCK
        assert bench.whole_slot_grid(kind, kv, 8192 << 20, 4) == 4096 * bench.COPY_BLOCK
        assert bench.whole_slot_grid(kind, lora, 8192 << 20, 4) == 12 * 320 * bench.COPY_BLOCK
    assert bench.whole_slot_grid("unpack", rr, 8192 << 20, 8) == 2048 * bench.COPY_BLOCK


def test_summarize_pmc_two_pools(tmp_path):
    # The LoRA workload's KV pool (whole-slot grid 4,096 workgroups) and
    # adapter pool (3,840): each pool's launches are told apart by their grid;
    # the kernel's ratio is over both pools' launches (bytes-weighted), each
    # pool's own under "pools".
    import bench
    pack, unpack = list(bench.PMC_KERNELS)
    kib = bench.PROBE_BYTES / 1024
    kv_kib = 512 * (2 << 20) / 1024
    lora_kib = 12 * 83886080 / 1024
    g_kv, g_lora = 4096 * bench.COPY_BLOCK, 3840 * bench.COPY_BLOCK
    hdr = ["Kernel_Name", "Counter_Name", "Counter_Value", "Grid_Size"]
    fetch, write = [(bench.PROBE_KERNEL, "FETCH_SIZE", kib, 1 << 20)], \
        [(bench.PROBE_KERNEL, "WRITE_SIZE", kib, 1 << 20)]
    for k in (pack, unpack):
        fetch += [(k, "FETCH_SIZE", kv_kib, g_kv), (k, "FETCH_SIZE", kv_kib, g_kv),
                  (k, "FETCH_SIZE", 1.02 * lora_kib, g_lora), (k, "FETCH_SIZE", 3.0, 1024)]
        write += [(k, "WRITE_SIZE", kv_kib, g_kv), (k, "WRITE_SIZE", kv_kib, g_kv),
                  (k, "WRITE_SIZE", 1.02 * lora_kib, g_lora), (k, "WRITE_SIZE", 3.0, 1024)]
    _write_csv(tmp_path / "f.csv", hdr, fetch)
    _write_csv(tmp_path / "w.csv", hdr, write)
    out = bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "zipf_lora",
                              str(tmp_path / "pmc.json"), ["cmd"])
    for short in ("pack", "unpack"):
        k = out["kernels"][short]
        assert k["dispatches"] == 3
        assert k["pools"]["kv"]["units_per_launch"] == 512
        assert k["pools"]["lora"]["units_per_launch"] == 12
        assert abs(k["pools"]["kv"]["traffic_over_algorithmic"] - 1.0) < 1e-12
        assert abs(k["pools"]["lora"]["traffic_over_algorithmic"] - 1.02) < 1e-12
        a_kv, a_lora = 2 * 2 * kv_kib * 1024, 2 * lora_kib * 1024
        want = (a_kv + 1.02 * a_lora) / (a_kv + a_lora)
        assert abs(k["traffic_over_algorithmic"] - want) < 1e-12
