#!/usr/bin/env python3
"""Benchmark of one simulation step of the invocation-distance memory manager
on one MI355X: plan (distances + activation mask -> victims, loads, block
table), evict (pack + device-to-host copy) and prefetch (host-to-device copy
+ unpack), on the 50,000-agent diffusion workload (one 160 GB pool) by
default.

Prints one JSON line.  ``value`` is evict+prefetch bytes moved per second of
wall time over the timed steps (inputs -- the per-step distances and masks --
already resident in HBM; the host link is part of the measured work).
``roofline`` is the dominant copy kernel against HBM peak, ``dma`` the copies
against the measured host-link bandwidth, ``plan_latency_us`` the plan call,
and ``cpu_baseline`` the CPU oracle on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0         # MI355X HBM3E, published
WORKLOAD_TEXT = {
    "tiny": "64 agents, 2x2x64 fp16 KV in 16 KiB pages, pool of 16 agents, 10% active/step",
    "roundrobin": "1,000 agents, 32x8x128 bf16 KV (128 KiB/token) in 2 MiB pages of 64 x 32 KiB, "
                  "prefix 512-2048 tokens, 40 GB pool, ~5% active/step round-robin, exact distances",
    "bursty": "10,000 agents, 2 MiB KV pages, lognormal prefixes, 120 GB pool, clustered bursts of "
              "1-3% per step, noisy distances",
    "zipf_lora": "2,000 agents, rank-16 LoRA (80 MiB, 448 planes, 256 slots) + 512-token KV "
                 "(30 GB pool), Zipf(1.1) activation 4%/step",
    "diffusion": "50,000 agents, unified 160 GB pool of 512 KiB units (KV pages + LoRA), "
                 "activation by messages on a degree-8 graph, noisy distances",
}


PMC_KERNELS = {"void ss::k_copy<true>(ss::CopyArgs)": "pack",
               "void ss::k_copy<false>(ss::CopyArgs)": "unpack"}
PROBE_KERNEL = "ss::k_probe_copy(char*, char const*, unsigned long long)"
PROBE_BYTES = 2 << 30          # bytes read and written by the probe copy (see probes())
COPY_ITEM_BYTES = 32768        # largest piece one wave copies (kItemBytes in the library)
COPY_BLOCK = 512               # threads per copy block (kCopyThreads)


def kernel_source_hash():
    """Hash of the copy kernels' source (the section between the "pack /
    unpack" and "launchers" headers of ss_kernels.hip)."""
    p = os.path.join(ROOT, "paper_2601_21473_amd", "csrc", "ss_kernels.hip")
    text = open(p).read()
    a = text.index("// pack / unpack")
    b = text.index("// launchers")
    return hashlib.sha256(text[a:b].encode()).hexdigest()[:16]


def launch_units(kind, blocks, n_items, n_planes):
    """Units one copy launch of ``blocks`` workgroups covers: the pack, and the
    unpack of pools whose chunks hold several items, take ceil(n_items / 8)
    workgroups per unit; the unpack of pools with one item per plane (run
    order) takes n_items workgroups per 8 units (the last group may be
    partial, so this is an upper bound there)."""
    waves = COPY_BLOCK // 64
    groups = (n_items + waves - 1) // waves
    if kind == "pack" or n_items != n_planes:
        return blocks // groups
    return blocks // n_items * waves


def whole_slot_grid(kind, spec, staging_bytes, ring):
    """Threads of a copy launch over one whole staging slot of pool ``spec``
    (each half of the staging buffer is cut into ``ring`` slots of whole
    units): the inverse of launch_units."""
    ups = (staging_bytes // 2 // ring) // spec.unit_bytes
    n_items = sum((c + COPY_ITEM_BYTES - 1) // COPY_ITEM_BYTES for c in spec.chunk_bytes)
    waves = COPY_BLOCK // 64
    if kind == "pack" or n_items != len(spec.chunk_bytes):
        blocks = ups * ((n_items + waves - 1) // waves)
    else:
        blocks = (ups + waves - 1) // waves * n_items
    return blocks * COPY_BLOCK


def summarize_pmc(fetch_csv, write_csv, workload, out_json, commands,
                  staging_bytes=8192 << 20, ring=4):
    """HBM traffic of the copy kernels from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE in KiB per dispatch), each scaled by the ratio of
    known bytes to the same counter on the probe's plain copy of PROBE_BYTES.
    Counted over the launches that cover a whole staging slot of a pool,
    recognised by their grid (whole_slot_grid; the pools of one workload
    must differ in it), whose unit count follows from the grid: pack
    launches item_groups blocks per unit, unpack n_items blocks per 8 units.
    With several pools, each kernel's ratio is over all of their whole-slot
    launches, with each pool's figures under "pools"."""
    import csv
    import collections
    import workloads as W
    pools = W.make_trace(workload, 0).pools
    vals = {}
    for path, counter in ((fetch_csv, "FETCH_SIZE"), (write_csv, "WRITE_SIZE")):
        per = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                per[r["Kernel_Name"]].append((float(r["Counter_Value"]), int(r["Grid_Size"])))
        vals[counter] = per
    factor = {c: PROBE_BYTES / 1024 / np.mean([v for v, _ in vals[c][PROBE_KERNEL]])
              for c in vals}
    out = {"workload": workload, "kernel_source_sha256_16": kernel_source_hash(),
           "commands": commands, "probe_scale_factor": factor, "kernels": {}}
    for name, short in PMC_KERNELS.items():
        grids = [whole_slot_grid(short, spec, staging_bytes, ring) for spec in pools]
        if len(set(grids)) != len(grids):
            raise ValueError(f"{workload}: pools with the same whole-slot {short} grid")
        per_pool = {}
        for spec, grid in zip(pools, grids):
            f = [v for v, g in vals["FETCH_SIZE"].get(name, []) if g == grid]
            w = [v for v, g in vals["WRITE_SIZE"].get(name, []) if g == grid]
            if not f or not w:
                continue
            n_items = sum((c + COPY_ITEM_BYTES - 1) // COPY_ITEM_BYTES for c in spec.chunk_bytes)
            units = launch_units(short, grid // COPY_BLOCK, n_items, len(spec.chunk_bytes))
            alg = 2 * units * spec.unit_bytes
            fetch_b = np.mean(f) * 1024 * factor["FETCH_SIZE"]
            write_b = np.mean(w) * 1024 * factor["WRITE_SIZE"]
            per_pool[spec.name] = {
                "dispatches": len(f), "grid_threads": grid, "units_per_launch": units,
                "hbm_read_bytes_per_launch": fetch_b, "hbm_write_bytes_per_launch": write_b,
                "hbm_bytes_per_launch": fetch_b + write_b,
                "algorithmic_bytes_per_launch": float(alg),
                "traffic_over_algorithmic": (fetch_b + write_b) / float(alg)}
        if len(pools) == 1:
            if per_pool:
                out["kernels"][short] = per_pool[pools[0].name]
        elif per_pool:
            hbm = sum(p["hbm_bytes_per_launch"] * p["dispatches"] for p in per_pool.values())
            alg = sum(p["algorithmic_bytes_per_launch"] * p["dispatches"] for p in per_pool.values())
            out["kernels"][short] = {
                "dispatches": sum(p["dispatches"] for p in per_pool.values()),
                "traffic_over_algorithmic": hbm / alg, "pools": per_pool}
    json.dump(out, open(out_json, "w"), indent=1)
    return out


def summarize_trace(trace_csv, out_md, title, command, note="", workload=None):
    """Markdown table of per-kernel launch counts and durations from a
    rocprofv3 --kernel-trace CSV (every kernel, plus the copy kernels split
    into full-slot launches and the rest).  With ``workload``, also each copy
    kernel's algorithmic bytes over all its launches (units per launch from
    the grid) divided by its summed durations, the figure ``roofline`` gives
    from HIP events."""
    import csv
    import collections
    rows = list(csv.DictReader(open(trace_csv)))
    per = collections.defaultdict(list)
    full = collections.defaultdict(list)
    top = collections.Counter()
    for r in rows:
        n = r["Kernel_Name"]
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        per[n].append(us)
        if n in PMC_KERNELS:
            top[(n, int(r["Grid_Size_X"]))] += 1
    grid_full = {n: max((g for (k, g) in top if k == n), default=0) for n in PMC_KERNELS}
    for r in rows:
        n = r["Kernel_Name"]
        if n in PMC_KERNELS and int(r["Grid_Size_X"]) == grid_full[n]:
            full[n].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    lines = [f"# {title}", "", "Command (repository root = `$REPO`, on one MI355X):", "",
             f"    {command}", "", f"Summary of `{os.path.basename(trace_csv)}` written by "
             f"`python bench.py --summarize-trace`.", "",
             "| Kernel | Calls | Total ms | Avg us | Min us | Max us |", "|---|---|---|---|---|---|"]
    for n, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        short = n.replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")
        lines.append(f"| `{short}` | {len(v)} | {sum(v) / 1e3:.2f} | {np.mean(v):.1f} | "
                     f"{min(v):.1f} | {max(v):.1f} |")
    lines += ["", "Copy kernels, launches over a whole staging slot (largest grid):", "",
              "| Kernel | Grid (threads) | Calls | Avg us | Median us | Min us |", "|---|---|---|---|---|---|"]
    for n, v in full.items():
        lines.append(f"| `{PMC_KERNELS[n]}` | {grid_full[n]:,} | {len(v)} | {np.mean(v):.1f} | "
                     f"{np.median(v):.1f} | {min(v):.1f} |")
    if workload:
        import workloads as W
        spec = W.make_trace(workload, 0).pools[0]
        n_items = sum((c + COPY_ITEM_BYTES - 1) // COPY_ITEM_BYTES for c in spec.chunk_bytes)
        lines += ["", f"Copy kernels over all launches ({workload} layout: {spec.unit_bytes:,} B "
                  f"units, {n_items} items per unit; algorithmic bytes = 2 x units x unit bytes, "
                  "units from the grid):", "",
                  "| Kernel | Launches | Algorithmic GB | Summed us | Achieved TB/s | Of 8 TB/s |",
                  "|---|---|---|---|---|---|"]
        for n, short in PMC_KERNELS.items():
            alg = us = 0.0
            k = 0
            for r in rows:
                if r["Kernel_Name"] != n:
                    continue
                blocks = int(r["Grid_Size_X"]) // COPY_BLOCK
                alg += 2.0 * launch_units(short, blocks, n_items, len(spec.chunk_bytes)) * \
                    spec.unit_bytes
                us += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
                k += 1
            if k:
                tbs = alg / us / 1e6
                lines.append(f"| `{short}` | {k} | {alg / 1e9:.1f} | {us:,.0f} | {tbs:.2f} | "
                             f"{tbs / 8.0:.3f} |")
    if note:
        lines += ["", note]
    open(out_md, "w").write("\n".join(lines) + "\n")
    return "\n".join(lines)


def summarize_copies(copy_csv, steps_jsonl, bench_json, out_md, title, command):
    """Host-link summary from a rocprofv3 --memory-copy-trace CSV.  The trace
    holds no sizes, so bytes come from the benchmark's per-step record of the
    same run (``--jsonl``): every staged step's written-back bytes crossed
    device to host, its loaded bytes host to device.  The step copies are those
    on the stream with the most copies of each direction (the pool's pair;
    the probes use streams of their own).  Per direction: copies, mean
    duration, busy time (union of the copies' intervals) and bytes / busy time
    against the one-way probe of the same run; both directions together:
    bytes / the union of all their intervals against the two-way probe."""
    import csv
    import collections
    rows = list(csv.DictReader(open(copy_csv)))
    recs = [json.loads(l) for l in open(steps_jsonl) if l.strip()]
    bench = json.loads([l for l in open(bench_json) if l.strip().startswith("{")][-1])
    probe = bench.get("probe") or {}
    by = collections.defaultdict(list)
    for r in rows:
        d = r["Direction"].replace("MEMORY_COPY_", "")
        by[(d, r["Stream_Id"])].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))

    def union(iv):
        iv = sorted(iv)
        tot, cs, ce = 0, None, None
        for a, b in iv:
            if ce is None or a > ce:
                if ce is not None:
                    tot += ce - cs
                cs, ce = a, b
            else:
                ce = max(ce, b)
        return tot + (ce - cs if ce is not None else 0)

    step_bytes = {"DEVICE_TO_HOST": sum(r["bytes_out"] - r.get("direct_out_bytes", 0) for r in recs),
                  "HOST_TO_DEVICE": sum(r["bytes_in"] - r.get("direct_in_bytes", 0) for r in recs)}
    one_way = {"DEVICE_TO_HOST": probe.get("d2h_GBps"), "HOST_TO_DEVICE": probe.get("h2d_GBps")}
    lines = [f"# {title}", "", "Command (repository root = `$REPO`, on one MI355X):", "",
             f"    {command}", "",
             f"Summary of `{os.path.basename(copy_csv)}` and of the per-step record "
             f"`{os.path.basename(steps_jsonl)}` ({len(recs)} steps: warm-up, timed and "
             "plan-latency steps) written by `python bench.py --summarize-copies`.  Bytes are "
             "the steps' staged write-back and load bytes; the probes' copies run on streams "
             "of their own and are left out.", "",
             "| Direction | Copies | Mean us | Median gap us | Busy ms | GB | GB/s while busy | "
             "One-way probe GB/s | Of probe |", "|---|---|---|---|---|---|---|---|---|"]
    all_iv = []
    out = {}
    for d in ("DEVICE_TO_HOST", "HOST_TO_DEVICE"):
        cands = [(len(v), k) for k, v in by.items() if k[0] == d]
        if not cands:
            continue
        _, key = max(cands)
        iv = by[key]
        all_iv += iv
        busy = union(iv) / 1e9
        mean_us = np.mean([b - a for a, b in iv]) / 1e3
        sv = sorted(iv)
        # idle time between successive copies of the stream, within a step
        gaps = [sv[i][0] - sv[i - 1][1] for i in range(1, len(sv))
                if 0 <= sv[i][0] - sv[i - 1][1] < 1_000_000]
        gap_us = float(np.median(gaps)) / 1e3 if gaps else float("nan")
        gb = step_bytes[d] / 1e9
        rate = gb / busy if busy else 0.0
        pw = one_way[d]
        out[d] = rate
        lines.append(f"| {d.replace('_', ' ').lower()} | {len(iv):,} | {mean_us:.1f} | {gap_us:.1f} | "
                     f"{1e3 * busy:,.1f} | {gb:.2f} | {rate:.1f} | "
                     f"{pw:.1f} | {rate / pw:.3f} |" if pw else
                     f"| {d} | {len(iv):,} | {mean_us:.1f} | {gap_us:.1f} | {1e3 * busy:,.1f} | "
                     f"{gb:.2f} | {rate:.1f} | - | - |")
    busy_all = union(all_iv) / 1e9
    tot = sum(step_bytes.values()) / 1e9
    dup = probe.get("duplex_GBps")
    lines += ["", f"Both directions: {tot:.2f} GB over {1e3 * busy_all:,.1f} ms in which at least "
              f"one direction copied = {tot / busy_all:.1f} GB/s" +
              (f" against the two-way probe's {dup:.1f} GB/s ({tot / busy_all / dup:.3f})."
               if dup else "."),
              "", f"Benchmark line of the same run: value {bench.get('value', 0):.1f} GB/s "
              f"(wall time of the timed steps), dma.frac_of_measured_link "
              f"{(bench.get('dma') or {}).get('frac_of_measured_link', float('nan')):.3f}."]
    open(out_md, "w").write("\n".join(lines) + "\n")
    return "\n".join(lines)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="diffusion", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--threshold", type=int, default=0xFFFFFFFF)
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--staging-mib", type=int, default=8192)
    ap.add_argument("--ring", type=int, default=4)
    ap.add_argument("--host-copies", type=int, default=128,
                    help="distinct host copies shared round-robin by agents; 0 = one per agent")
    ap.add_argument("--plan-steps", type=int, default=20)
    ap.add_argument("--null-stream", action="store_true",
                    help="queue the plan and the step on the null stream instead of a stream "
                         "of the caller's own")
    ap.add_argument("--blocking-wait", action="store_true",
                    help="the pools' waits (ss_sync) block instead of polling "
                         "(SS_FLAG_POLL_WAIT off)")
    ap.add_argument("--direct-mib", type=float, default=4,
                    help="directions of a step that move at most this many MiB go by kernel "
                         "straight between units and host copies (0 = always staged)")
    ap.add_argument("--cpu-steps", type=int, default=4)
    ap.add_argument("--cpu-agents", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="sample steps until the CPU oracle's timed work reaches this")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", action="store_true")
    ap.add_argument("--clean-evict", action="store_true",
                    help="mark every agent's memory unchanged: evictions release units "
                         "without writing back (write-back elision)")
    ap.add_argument("--no-objects", action="store_true",
                    help="skip the shared-object distance kernel measurement")
    ap.add_argument("--objects-only", action="store_true",
                    help="only the shared-object distance measurement (for profiling)")
    ap.add_argument("--no-estimators", action="store_true",
                    help="skip the distance estimator measurements")
    ap.add_argument("--estimators-only", action="store_true",
                    help="only the distance estimator measurements (for profiling)")
    ap.add_argument("--no-loader", action="store_true",
                    help="skip the load-task scheduler measurement")
    ap.add_argument("--loader-only", action="store_true",
                    help="only the load-task scheduler measurement")
    ap.add_argument("--objects-trees", type=int, default=160)
    ap.add_argument("--objects-agents", type=int, default=50_000)
    ap.add_argument("--objects-depth", type=int, default=5)
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "OUT_JSON"),
                    help="write the copy kernels' HBM traffic from two rocprofv3 --pmc runs")
    ap.add_argument("--pmc-commands", nargs="*", default=[])
    ap.add_argument("--summarize-trace", nargs=4, metavar=("TRACE_CSV", "OUT_MD", "TITLE", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --kernel-trace CSV (with "
                         "--workload: the copy kernels' achieved rate over all launches too)")
    ap.add_argument("--trace-workload", default=None,
                    help="workload whose unit layout --summarize-trace uses for the copy kernels")
    ap.add_argument("--summarize-copies", nargs=6,
                    metavar=("COPY_CSV", "STEPS_JSONL", "BENCH_JSON", "OUT_MD", "TITLE", "COMMAND"),
                    help="write a host-link summary of a rocprofv3 --memory-copy-trace CSV")
    ap.add_argument("--jsonl", default=None,
                    help="write one JSON record per step (warm-up, timed and plan-latency steps) "
                         "to this file: the plan's counts and bytes and the host time of the "
                         "step's calls (no extra waits)")
    ap.add_argument("--jsonl-timing", action="store_true",
                    help="with --jsonl, add each step's plan, pack, copy and unpack times from "
                         "the pools' timing counters (the host then waits for every step before "
                         "queueing the next)")
    return ap.parse_args()


def probes(binding, host=None):
    """Plain-copy HBM probe and pinned host-link probes (1 GiB copies: H2D,
    D2H and both at once).  ``host`` is pinned memory of at least 2 GiB to
    probe against (the pool's own host copies, so that the link is measured
    to the memory the workload moves); without it a fresh pinned buffer is
    used, whose NUMA placement may differ from the pool's."""
    from paper_2601_21473_amd.memory import DeviceBuffer, HostBuffer
    out = {}
    n = 2 << 30
    a, b = DeviceBuffer(n), DeviceBuffer(n)
    ms = binding.probe_copy(b.ptr, a.ptr, n, iters=10)
    out["hbm_copy_GBps"] = 2 * n / ms / 1e6
    # the runtime's own device-to-device copy of the same buffers, for
    # reference (it may return before the copy ends: each is followed by a
    # wait for the null stream; best host wall time of five)
    walls = []
    for _ in range(5):
        t0 = time.perf_counter()
        binding.copy(b.ptr, a.ptr, n)
        binding.null_stream_sync()
        walls.append(time.perf_counter() - t0)
    out["runtime_dtod_copy_GBps"] = 2 * n / min(walls) / 1e9
    a.free()
    b.free()
    m = 1 << 30
    own = host is None or host.nbytes < 2 * m
    h = HostBuffer(2 * m) if own else host
    d = DeviceBuffer(2 * m)
    if own:
        h.np[:] = 1                              # host pages resident before timing
    # best of three trials of five copies each, per direction
    best = lambda direction: min(binding.probe_link(h.ptr, d.ptr, m, direction, 5)
                                 for _ in range(3))
    out["h2d_GBps"] = m / best(0) / 1e6
    out["d2h_GBps"] = m / best(1) / 1e6
    out["duplex_GBps"] = 2 * m / best(2) / 1e6
    out["host_memory"] = "fresh pinned buffer" if own else "the pool's pinned host copies"
    if own:
        h.free()
    d.free()
    return out


OBJ_BRANCH = 8                   # prefix trees of the shared-object measurement


def object_bench(args, binding, W, DeviceBuffer):
    """Shared-object distances (Appendix A, fine-grained distance assignment)
    on a prefix forest: ``objects-trees`` simulations of ``objects-agents``
    agents (default 160 x 50,000, the diffusion workload's agent count), each
    sharing a branching-8 prefix tree of ``objects-depth`` levels with one
    private leaf per agent, agents spread uniformly over the tree; 1% of agents
    active, distances uniform in [1, 2^20).  Also the latency at 16,384 agents
    and the oracle's rate on that small map."""
    def measure(off, agents, n, iters, rng):
        M, R = len(off) - 1, int(off[-1])
        D = rng.integers(1, 1 << 20, size=n).astype(np.uint32)
        act = (rng.random(n) < 0.01).astype(np.uint8)
        bufs = [DeviceBuffer(4 * (M + 1)), DeviceBuffer(4 * R), DeviceBuffer(4 * n),
                DeviceBuffer(n), DeviceBuffer(4 * M), DeviceBuffer(M)]
        wsb = binding.object_distances_workspace(M, R, n)
        ws = DeviceBuffer(wsb)
        for b, a in zip(bufs, [off.astype(np.uint32), agents, D, act]):
            b.upload(a)
        ms = binding.probe_object_distances(bufs[0].ptr, bufs[1].ptr, M, R, bufs[2].ptr,
                                            bufs[3].ptr, n, bufs[4].ptr, bufs[5].ptr, ws.ptr,
                                            wsb, iters)
        for b in bufs + [ws]:
            b.free()
        alg = 4 * (M + 1) + 4 * R + 5 * n + 5 * M
        return M, R, ms, alg, (D, act)

    rng = np.random.default_rng(args.seed + 17)
    off, agents, _ = W.prefix_forest(args.objects_trees, args.objects_agents, OBJ_BRANCH,
                                     args.objects_depth, seed=args.seed)
    n = args.objects_trees * args.objects_agents
    M, R, ms, alg, _ = measure(off, agents, n, 20, rng)
    del off, agents
    small_off, small_agents, _ = W.prefix_tree_objects(16384, 4, 6, seed=args.seed)
    m2, r2, ms2, alg2, (D2, act2) = measure(small_off, small_agents, 16384, 200, rng)
    out = {"workload": f"{args.objects_trees} prefix trees x {args.objects_agents} agents, "
                       f"branching {OBJ_BRANCH}, depth {args.objects_depth}, private leaves; "
                       "1% active, distances uniform in [1, 2^20)",
           "objects": M, "refs": R, "agents": n,
           "kernels": "k_obj_prep + k_obj_min + k_obj_fix (event time of the three)",
           "us_per_call": 1e3 * ms, "algorithmic_bytes": alg,
           "roofline": {"bound": "hbm", "achieved": alg / ms / 1e6, "peak": HBM_PEAK_GBPS,
                        "unit": "GB/s", "frac": alg / ms / 1e6 / HBM_PEAK_GBPS, "traffic": None},
           "small": {"agents": 16384, "objects": m2, "refs": r2, "us_per_call": 1e3 * ms2,
                     "GBps": alg2 / ms2 / 1e6}}
    if not args.no_cpu_baseline:
        from oracle.objects import object_distances
        t0 = time.perf_counter()
        object_distances(small_off, small_agents, D2, act2)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": m2 / dt, "unit": "objects/s", "cores": 1,
                               "kind": "oracle", "sample": f"the 16,384-agent map ({m2} objects)",
                               "gpu_objects_per_s": M / (ms * 1e-3)}
    return out


VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12   # 32-bit VALU lane-instructions/s, MI355X
PAIR_VALU = 2.5                # packed subtract + dot2 + half a min3 per pair (k_pair_min)


def estimator_bench(args, binding, W, DeviceBuffer):
    """Distance estimators of Section 3.2: hop counts on the diffusion
    workload's graph (50,000 agents, out-degree 8, sources = the agents
    active at step 10) and on a 4M-vertex out-degree-8 random graph from 1%
    sources; interaction distances of 10,000 and 50,000 agents on a
    2048 x 2048 tile grid."""
    rng = np.random.default_rng(args.seed + 23)
    out = {}

    def timed(fn, iters):
        t = binding.EventTimer()
        try:
            fn(t.handle)                       # warm-up
            with t:
                for _ in range(iters):
                    fn(t.handle)
            return t.ms / iters
        finally:
            t.close()

    def hops_case(off, col, src, label, iters):
        V, E = len(off) - 1, len(col)
        b = [DeviceBuffer(4 * (V + 1)), DeviceBuffer(max(4, 4 * E)), DeviceBuffer(max(4, 4 * len(src))),
             DeviceBuffer(4 * V)]
        wsb = binding.hop_distances_workspace(V)
        ws = DeviceBuffer(wsb)
        b[0].upload(np.asarray(off, np.uint32))
        b[1].upload(np.asarray(col, np.uint32))
        b[2].upload(np.asarray(src, np.uint32))
        ms = timed(lambda st: binding.hop_distances(b[0].ptr, b[1].ptr, V, E, b[2].ptr, len(src),
                                                    0xFFFFFFFF, b[3].ptr, ws.ptr, wsb, st), iters)
        h = b[3].download(0, 4 * V).view(np.uint32)
        reached = h != 0xFFFFFFFF
        deg = np.diff(np.asarray(off, np.int64))
        traversed = int(deg[reached].sum())
        levels = int(h[reached].max()) if reached.any() else 0
        for x in b + [ws]:
            x.free()
        alg = 4 * (V + 1) + 4 * E + 20 * V
        return {"graph": label, "vertices": V, "edges": E, "sources": len(src), "levels": levels,
                "us_per_call": 1e3 * ms, "edges_traversed": traversed,
                "GTEPS": traversed / ms / 1e6, "algorithmic_bytes": alg,
                "GBps": alg / ms / 1e6, "hbm_frac": alg / ms / 1e6 / HBM_PEAK_GBPS}

    tr = W.make_trace("diffusion", args.seed)
    nb = tr.meta["out_neighbors"]
    V = nb.shape[0]
    out["hops_diffusion"] = hops_case(np.arange(0, 8 * V + 1, 8), nb.reshape(-1),
                                      np.flatnonzero(tr.active[10]),
                                      "diffusion workload graph (50,000 x out-degree 8)", 50)
    V2 = 4_000_000
    col = rng.integers(0, V2, size=8 * V2).astype(np.uint32)
    out["hops_large"] = hops_case(np.arange(0, 8 * V2 + 1, 8), col,
                                  rng.choice(V2, V2 // 100, replace=False),
                                  "random 4,000,000 x out-degree 8", 10)
    del col

    for n in (10_000, 50_000):
        pos = rng.integers(0, 2048, size=(n, 2)).astype(np.int32)
        d_act = rng.integers(0, 100, size=n).astype(np.uint32)
        b = [DeviceBuffer(8 * n), DeviceBuffer(4 * n), DeviceBuffer(4 * n)]
        wsb = binding.interaction_distances_workspace(n)
        ws = DeviceBuffer(wsb)
        b[0].upload(pos.reshape(-1))
        b[1].upload(d_act)
        ms = timed(lambda st: binding.interaction_distances(b[0].ptr, b[1].ptr, n, 3, 2, b[2].ptr,
                                                            ws.ptr, wsb, st), 20)
        for x in b + [ws]:
            x.free()
        pairs = n * (n - 1)
        ach = pairs * PAIR_VALU / ms / 1e9
        out[f"interaction_{n}"] = {
            "agents": n, "grid": "2048 x 2048 tiles", "velocity": 3, "radius": 2,
            "us_per_call": 1e3 * ms, "Gpairs_per_s": pairs / ms / 1e6,
            "roofline": {"bound": "alu", "achieved": ach, "peak": VALU_PEAK_TOPS,
                         "unit": "T VALU lane-instructions/s", "frac": ach / VALU_PEAK_TOPS,
                         "per_pair": PAIR_VALU}}
    return out


LOADER_AGENTS = 128             # background load tasks of the scheduler measurement
LOADER_URGENT = 8               # urgent (distance 0) arrivals timed per configuration


def loader_bench(args, binding, W, spec0, PoolMemory, DeviceBuffer, probe):
    """Load-task scheduler (Appendix A, load task scheduler and preemption
    support) on the round-robin workload's module layout (2 MiB units of
    64 x 32 KiB, agents of 32-128 units): for chunks of 4, 16 and 64 units
    (8, 32 and 128 MiB; ring of 4 staging slots, so 4 chunks in flight)

    * load rate: 128 queued tasks drained in distance order, bytes per second
      of wall time against the measured one-way host-to-device rate;
    * preemption latency: with the window full of a running task's chunks, a
      distance-0 task arrives; time from its submission until all its units
      have landed, with preemption and with preemption off (the running
      task finishes first), median over 8 arrivals, next to the time its
      own bytes need on the link.

    ``spec0`` is the round-robin workload's pool; the module holds its first
    136 agents.  Destination units are a seeded permutation of the module's
    units (each task's units scattered over the pool)."""
    n_agents = LOADER_AGENTS + LOADER_URGENT
    units = np.asarray(spec0.agent_units[:n_agents], dtype=np.uint32)
    cap = int(units.sum())
    spec = W.PoolSpec("loader", cap, list(spec0.chunk_bytes), units)
    ub = spec.unit_bytes
    rng = np.random.default_rng(args.seed)
    perm = rng.permutation(cap).astype(np.int32)
    off = np.concatenate([[0], np.cumsum(units)]).astype(np.int64)
    dist_bg = rng.permutation(np.arange(2, 2 + LOADER_AGENTS)).astype(np.uint32)
    h2d = probe.get("h2d_GBps") if probe else None
    out = {"module": "round-robin layout: 2 MiB units of 64 x 32 KiB, agents of 32-128 units",
           "tasks": LOADER_AGENTS, "task_bytes": int(units[:LOADER_AGENTS].sum()) * ub,
           "window_chunks": 4, "configs": []}
    for chunk_units in (4, 16, 64):
        mem = PoolMemory(spec, 4 * chunk_units * ub, 4, host_slots=16)
        mem.host_np[:] = 1                    # host pages resident before timing
        dl = DeviceBuffer(perm.nbytes)
        dl.upload(perm)
        ptr = lambda a: dl.ptr + 4 * int(off[a])
        rec = {"chunk_units": chunk_units, "chunk_bytes": chunk_units * ub}
        try:
            for preempt in (True, False):
                L = binding.Loader([mem.desc_args()], preempt=preempt)
                try:
                    if preempt:
                        # load rate: drain every background task
                        L.submit([(0, a, int(dist_bg[a]), ptr(a)) for a in range(LOADER_AGENTS)])
                        t0 = time.perf_counter()
                        L.pump(1 << 16)
                        L.sync()
                        wall = time.perf_counter() - t0
                        rec["load_GBps"] = out["task_bytes"] / wall / 1e9
                        if h2d:
                            rec["frac_of_measured_h2d"] = rec["load_GBps"] / h2d
                    L.submit([(0, a, int(dist_bg[a]), ptr(a)) for a in range(LOADER_AGENTS)])
                    L.pump(4)                 # window full
                    lat, own = [], []
                    for k in range(LOADER_URGENT):
                        ua = LOADER_AGENTS + k
                        L.pump(4)
                        t0 = time.perf_counter()
                        L.submit([(0, ua, 0, ptr(ua))])
                        done = False
                        while not done:
                            got = L.pump(1)
                            assert got, "urgent task was not scheduled"
                            done = any(a == ua and f & binding.SS_LOAD_DONE
                                       for (_, a, _, _, f) in got)
                        L.sync()
                        lat.append(time.perf_counter() - t0)
                        own.append(int(units[ua]) * ub)
                    key = "preempt" if preempt else "no_preempt"
                    rec[f"urgent_latency_ms_{key}"] = 1e3 * float(np.median(lat))
                    if preempt:
                        rec["preemptions"] = L.stats()["preemptions"]
                        if h2d:
                            rec["urgent_own_bytes_ms"] = 1e3 * float(np.median(own)) / h2d / 1e9
                finally:
                    L.close()
        finally:
            dl.free()
            mem.free()
        out["configs"].append(rec)
    return out


CPU_POOL_WINDOW = 1024            # units of the oracle's byte pool in the CPU baseline


def cpu_baseline(trace, warmup, n_steps, n_agents_moved, threshold, budget, min_seconds=0.0):
    """The CPU oracle on a bounded sample: the oracle plan for every agent on
    steps [warmup, warmup + n_steps) (after replaying the earlier steps'
    plans), and the oracle's numpy gather/scatter of the bytes of the first
    ``n_agents_moved`` written-back victims and loads of each sampled step
    through warm buffers.  Sampling goes on past ``n_steps`` steps until the
    timed work reaches ``min_seconds`` or the trace ends.  The moved units' rows are taken modulo a window of
    CPU_POOL_WINDOW units of the oracle's byte pool (same row-gather pattern,
    memory bounded to the window)."""
    from types import SimpleNamespace
    from oracle import OraclePool, BytePool, apply_step_bytes
    spec = trace.pools[0]
    ub = spec.unit_bytes
    opool = OraclePool(spec.capacity_units, spec.agent_units, ub)
    for t in range(warmup):
        opool.plan_step(trace.dist[t], trace.active[t], threshold, budget)
    window = min(spec.capacity_units, CPU_POOL_WINDOW)
    bp = BytePool(window, spec.chunk_bytes)
    for plane in bp.planes:
        plane[:] = 1                                  # pages resident before timing
    s = spec.agent_units.astype(np.int64)
    max_agent = int(s.max()) * ub
    stage_out = np.ones(n_agents_moved * max_agent, dtype=np.uint8)
    stage_in = np.ones(n_agents_moved * max_agent, dtype=np.uint8)
    host_out = np.ones(max_agent, dtype=np.uint8)     # one host copy written by every victim
    host_in = np.ones(max_agent, dtype=np.uint8)      # one host copy read by every load
    t_plan = t_move = 0.0
    moved = 0
    t = warmup
    while t < len(trace.dist) and (t < warmup + n_steps or t_plan + t_move < min_seconds):
        t0 = time.perf_counter()
        plan = opool.plan_step(trace.dist[t], trace.active[t], threshold, budget)
        t_plan += time.perf_counter() - t0
        V = plan.written[:n_agents_moved]
        Ld = plan.loads[:n_agents_moved]
        nvu = int(s[V].sum())
        nlu = int(s[Ld].sum())
        sub = SimpleNamespace(victims=V, written=V, loads=Ld,
                              victim_units=plan.written_units[:nvu] % window,
                              written_units=plan.written_units[:nvu] % window,
                              load_units=plan.load_units[:nlu] % window)
        t0 = time.perf_counter()
        apply_step_bytes(bp, sub, s, lambda a: host_in[:s[a] * ub],
                         lambda a, b: host_out[:len(b)].__setitem__(slice(None), b),
                         staging_out=stage_out, staging_in=stage_in)
        t_move += time.perf_counter() - t0
        moved += (nvu + nlu) * ub
        t += 1
    n_steps = t - warmup
    return {"value": moved / (t_plan + t_move) / 1e9, "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"steps {warmup}-{t - 1} of the {trace.name} trace: oracle plan "
                      f"of all {trace.n_agents} agents per step ({1e3 * t_plan / n_steps:.2f} ms/step) "
                      f"+ numpy gather/scatter of the first {n_agents_moved} written-back victims' "
                      f"and loads' bytes ({moved / 1e9:.2f} GB in {t_move:.2f} s; unit rows taken "
                      f"modulo a {window}-unit window of the byte pool), single thread",
            "host_threads_available": len(os.sched_getaffinity(0)), "cpu_model": cpu_model()}


def cpu_model() -> str:
    """The host CPU's model name as the kernel reports it (empty if unknown)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def main():
    args = parse()
    if args.summarize_trace:
        print(summarize_trace(*args.summarize_trace, workload=args.trace_workload))
        return
    if args.summarize_copies:
        print(summarize_copies(*args.summarize_copies))
        return
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(*args.summarize_pmc[:2], args.workload,
                                       args.summarize_pmc[2], args.pmc_commands,
                                       staging_bytes=args.staging_mib << 20, ring=args.ring),
                         indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested): the library "
              f"has no multi-GPU path; agents would shard across GPUs, each GPU planning "
              f"and moving its own agents with no exchange", file=sys.stderr)
        sys.exit(2)
    import workloads as W
    from paper_2601_21473_amd import binding
    from paper_2601_21473_amd.memory import DeviceBuffer, PoolMemory

    assert binding.device_count() > 0, "bench.py needs a GPU"
    if args.objects_only:
        print(json.dumps({"object_distances": object_bench(args, binding, W, DeviceBuffer)}),
              flush=True)
        return
    if args.estimators_only:
        print(json.dumps({"estimators": estimator_bench(args, binding, W, DeviceBuffer)}),
              flush=True)
        return
    if args.loader_only:
        rr = W.make_trace("roundrobin", 0).pools[0]
        pr = {} if args.no_probe else probes(binding)
        print(json.dumps({"loader": loader_bench(args, binding, W, rr, PoolMemory, DeviceBuffer,
                                                 pr), "probe": pr}), flush=True)
        return
    trace = W.make_trace(args.workload, args.seed)
    T_need = args.warmup + args.steps
    if T_need > trace.n_steps:
        sys.exit(f"warmup + steps = {T_need} exceeds the trace's {trace.n_steps} steps")
    budget = args.budget
    thr = args.threshold

    mems, pools = [], []
    for spec in trace.pools:
        host_slots = None if args.host_copies == 0 else args.host_copies
        mem = PoolMemory(spec, args.staging_mib << 20, args.ring, host_slots=host_slots)
        mems.append(mem)
        pools.append(mem.make_pool(timing=True, direct_bytes=int(args.direct_mib * (1 << 20)),
                                   poll_wait=not args.blocking_wait))
    probe = {} if args.no_probe else probes(binding, mems[0].host)
    N = trace.n_agents
    d_np = np.ascontiguousarray(trace.dist, dtype=np.uint32)
    a_np = np.ascontiguousarray(trace.active, dtype=np.uint8)
    dist, act = DeviceBuffer(d_np.nbytes), DeviceBuffer(a_np.nbytes)
    dist.upload(d_np)
    act.upload(a_np)
    # the caller's stream: a non-blocking stream of its own, as a serving loop
    # would use (--null-stream: the null stream, which adds the runtime's
    # cross-stream synchronization to every call queued on it)
    cstream = None if args.null_stream else binding.Stream()
    stream = 0 if cstream is None else cstream.handle
    clean = DeviceBuffer(N) if args.clean_evict else None
    if clean is not None:
        clean.upload(np.zeros(N, dtype=np.uint8))
    dirty_ptr = clean.ptr if clean is not None else 0

    def sync():
        for p in pools:
            p.sync()

    # per-step record (--jsonl): the step's plan, bytes and, from the pools'
    # timing counters, its plan, pack, copy and unpack times
    jl = open(args.jsonl, "w") if args.jsonl else None
    jl_prev = [None]
    stat_keys = ("pack_ms", "unpack_ms", "d2h_ms", "h2d_ms", "plan_gpu_ms", "direct_out_ms",
                 "direct_in_ms", "pack_launches", "unpack_launches", "direct_out_bytes",
                 "direct_in_bytes")

    def record(t, phase, plans, t_call):
        if jl is None:
            return
        direct = int(args.direct_mib * (1 << 20))
        out_b = sum(pl["bytes_out"] for pl in plans)
        in_b = sum(pl["bytes_in"] for pl in plans)
        rec = {"t": t, "phase": phase, "n_victims": sum(pl["n_victims"] for pl in plans),
               "n_loads": sum(pl["n_loads"] for pl in plans),
               "units_out": sum(pl["units_out"] for pl in plans),
               "units_in": sum(pl["units_in"] for pl in plans),
               "bytes_out": out_b, "bytes_in": in_b,
               # a direction at or below the direct limit moves by kernel, not by copies
               "direct_out_bytes": sum(pl["bytes_out"] for pl in plans
                                       if 0 < pl["bytes_out"] <= direct),
               "direct_in_bytes": sum(pl["bytes_in"] for pl in plans
                                      if 0 < pl["bytes_in"] <= direct),
               "t_step_call_ms": 1e3 * t_call}
        if args.jsonl_timing:
            cur = [p.stats() for p in pools]       # waits for the step
            tot = {k: sum(c[k] for c in cur) for k in stat_keys}
            tot["plan_host_us"] = sum(sum(c["plan_host_us"]) for c in cur)
            prev = jl_prev[0] or {k: 0 for k in tot}
            d = {k: tot[k] - prev[k] for k in tot}
            jl_prev[0] = tot
            rec.update({"t_plan_us": d["plan_host_us"], "t_plan_gpu_us": 1e3 * d["plan_gpu_ms"],
                        "t_pack_ms": d["pack_ms"], "t_d2h_ms": d["d2h_ms"],
                        "t_h2d_ms": d["h2d_ms"], "t_unpack_ms": d["unpack_ms"],
                        "t_direct_out_ms": d["direct_out_ms"],
                        "t_direct_in_ms": d["direct_in_ms"],
                        "pack_launches": d["pack_launches"],
                        "unpack_launches": d["unpack_launches"]})
        jl.write(json.dumps(rec) + "\n")

    def step(t, phase="timed"):
        ts = time.perf_counter()
        plans = [p.plan_step(dist.ptr + 4 * N * t, act.ptr + N * t, thr, budget, stream,
                             dirty_ptr, lists=False) for p in pools]
        for p in pools:
            p.evict_pack(stream)
        for p in pools:
            p.prefetch_unpack(stream)
        record(t, phase, plans, time.perf_counter() - ts)
        return plans

    # the first steps fill the empty pool: timed apart from the steady state
    fill_steps = min(10, args.warmup)
    fill_b = 0
    sync()
    tf = time.perf_counter()
    for t in range(args.warmup):
        plans = step(t, "warmup")
        if t < fill_steps:
            fill_b += sum(pl["bytes_out"] + pl["bytes_in"] for pl in plans)
        if t == fill_steps - 1:
            sync()
            fill_wall = time.perf_counter() - tf
    sync()
    for p in pools:
        p.reset_stats()
    moved = out_b = in_b = 0
    step_wall = []
    sync()
    t0 = time.perf_counter()
    for k in range(args.steps):
        ts = time.perf_counter()
        plans = step(args.warmup + k)
        step_wall.append(time.perf_counter() - ts)
        for pl in plans:
            out_b += pl["bytes_out"]
            in_b += pl["bytes_in"]
    sync()
    wall = time.perf_counter() - t0
    moved = out_b + in_b
    stats = [p.stats() for p in pools]

    # plan latency: each plan issued with the device idle (after the pools'
    # wait, which polls unless --blocking-wait: a launch after a blocking wait
    # on long work costs the host 2-3 times as much); wall time of the
    # Python call (counts only) and the library's own host time of the C call
    # (stats are read only after a plan, so that nothing is submitted between
    # the wait for the previous step and the measured call).  First with the
    # inputs in device memory, then with the same kind of inputs in host
    # memory (numpy arrays, copied by the call into pinned memory that the
    # plan kernel reads over the host link).  The latency steps follow the
    # timed ones and wrap around at the trace's end (any step's inputs are a
    # valid plan input).
    def plan_latency(host_inputs, first):
        lat, lat_c = [], []
        c_prev = sum(sum(p.stats()["plan_host_us"]) for p in pools)
        for k in range(args.plan_steps):
            sync()
            t = (first + k) % trace.n_steps
            if host_inputs:
                d_ptr, a_ptr = d_np[t].ctypes.data, a_np[t].ctypes.data
            else:
                d_ptr, a_ptr = dist.ptr + 4 * N * t, act.ptr + N * t
            ts = time.perf_counter()
            plans = [p.plan_step(d_ptr, a_ptr, thr, budget, stream, dirty_ptr, lists=False)
                     for p in pools]
            lat.append(time.perf_counter() - ts)
            c_now = sum(sum(p.stats()["plan_host_us"]) for p in pools)
            lat_c.append(c_now - c_prev)
            c_prev = c_now
            for p in pools:
                p.evict_pack(stream)
            for p in pools:
                p.prefetch_unpack(stream)
            record(t, "plan_host_inputs" if host_inputs else "plan", plans, lat[-1])
        sync()
        lat_us = np.array(lat) * 1e6
        return {"median": float(np.median(lat_us)), "p99": float(np.percentile(lat_us, 99)),
                "c_call_median": float(np.median(lat_c)),
                "c_call_p99": float(np.percentile(lat_c, 99))}

    lat_dev = plan_latency(False, args.warmup + args.steps)
    plan_stats = [p.stats() for p in pools]
    lat_host = plan_latency(True, args.warmup + args.steps + args.plan_steps)
    if jl is not None:
        jl.close()
    if probe:
        # a second probe after the timed steps: each direction keeps its better
        # reading
        again = probes(binding, mems[0].host)
        probe = {k: (max(v, again[k]) if isinstance(v, float) else v) for k, v in probe.items()}
    for p in pools:
        p.close()
    for m in mems:
        m.free()
    dist.free()
    if cstream is not None:
        cstream.close()
    act.free()
    if clean is not None:
        clean.free()

    pack_ms = sum(s["pack_ms"] for s in stats)
    unpack_ms = sum(s["unpack_ms"] for s in stats)
    pack_b = sum(s["pack_bytes"] for s in stats)
    unpack_b = sum(s["unpack_bytes"] for s in stats)
    pack_n = sum(s["pack_launches"] for s in stats)
    unpack_n = sum(s["unpack_launches"] for s in stats)
    kern = {
        "pack": {"launches": pack_n, "bytes_per_launch": 2 * pack_b / max(pack_n, 1),
                 "avg_us": 1e3 * pack_ms / max(pack_n, 1),
                 "GBps": 2 * pack_b / max(pack_ms, 1e-9) / 1e6},
        "unpack": {"launches": unpack_n, "bytes_per_launch": 2 * unpack_b / max(unpack_n, 1),
                   "avg_us": 1e3 * unpack_ms / max(unpack_n, 1),
                   "GBps": 2 * unpack_b / max(unpack_ms, 1e-9) / 1e6},
    }
    direct = {k: sum(s[k] for s in stats) for k in
              ("direct_out_launches", "direct_in_launches", "direct_out_bytes", "direct_in_bytes",
               "direct_out_ms", "direct_in_ms", "duplex_launches", "duplex_bytes", "duplex_ms")}
    for d in ("out", "in"):
        direct[f"direct_{d}_GBps"] = (direct[f"direct_{d}_bytes"] /
                                      max(direct[f"direct_{d}_ms"], 1e-9) / 1e6)
    direct["duplex_GBps"] = direct["duplex_bytes"] / max(direct["duplex_ms"], 1e-9) / 1e6
    dom = "pack" if pack_ms >= unpack_ms else "unpack"
    direct_ms = direct["direct_out_ms"] + direct["direct_in_ms"]
    if direct["duplex_ms"] > max(pack_ms + unpack_ms, direct_ms):
        # steps small enough to move both directions in one launch straight
        # over the host link: peak = the measured two-way copy-engine rate
        n = max(direct["duplex_launches"], 1)
        peak = probe.get("duplex_GBps") if probe else None
        ach = direct["duplex_GBps"]
        roofline = {"bound": "host-link", "kernel": "k_duplex", "achieved": ach, "peak": peak,
                    "unit": "GB/s", "frac": ach / peak if peak else None, "traffic": None,
                    "algorithmic_bytes_per_launch": direct["duplex_bytes"] / n}
    elif pack_ms + unpack_ms >= direct_ms:
        traffic = None
        pmc_path = os.path.join(ROOT, "profiles", f"k_copy_{args.workload}_pmc.json")
        if os.path.exists(pmc_path):
            pmc = json.load(open(pmc_path))
            ratio = pmc["kernels"].get(dom, {}).get("traffic_over_algorithmic")
            if pmc.get("kernel_source_sha256_16") == kernel_source_hash() and ratio:
                # HBM bytes per whole-slot launch over its algorithmic bytes,
                # applied to the timed launches' average size
                traffic = ratio * kern[dom]["bytes_per_launch"]
        roofline = {"bound": "hbm", "kernel": f"k_copy<{dom}>", "achieved": kern[dom]["GBps"],
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": kern[dom]["GBps"] / HBM_PEAK_GBPS, "traffic": traffic,
                    "algorithmic_bytes_per_launch": kern[dom]["bytes_per_launch"]}
    else:
        # steps small enough to move by kernel straight over the host link:
        # the dominant launches are host-link bound (peak: the measured one-way
        # copy-engine rate of the same direction)
        d = "out" if direct["direct_out_ms"] >= direct["direct_in_ms"] else "in"
        n = max(direct[f"direct_{d}_launches"], 1)
        peak = (probe.get("d2h_GBps" if d == "out" else "h2d_GBps") if probe else None)
        ach = direct[f"direct_{d}_GBps"]
        roofline = {"bound": "host-link", "kernel": f"k_copy<{'pack' if d == 'out' else 'unpack'}>"
                    " direct", "achieved": ach, "peak": peak, "unit": "GB/s",
                    "frac": ach / peak if peak else None, "traffic": None,
                    "algorithmic_bytes_per_launch": direct[f"direct_{d}_bytes"] / n}
    d2h_b = sum(s["d2h_bytes"] for s in stats)
    h2d_b = sum(s["h2d_bytes"] for s in stats)
    d2h_ms = sum(s["d2h_ms"] for s in stats)
    h2d_ms = sum(s["h2d_ms"] for s in stats)
    dma = {"bytes_d2h": d2h_b, "bytes_h2d": h2d_b,
           "d2h_GBps": d2h_b / max(d2h_ms, 1e-9) / 1e6, "h2d_GBps": h2d_b / max(h2d_ms, 1e-9) / 1e6,
           "wall_GBps": moved / wall / 1e9}
    if probe:
        # shortest time the measured link allows: each direction at its own
        # one-way rate, and both together at the measured two-way rate
        duplex = probe["duplex_GBps"] > 1.2 * max(probe["h2d_GBps"], probe["d2h_GBps"])
        one_way = max(out_b / probe["d2h_GBps"], in_b / probe["h2d_GBps"])
        ideal = (max(one_way, (out_b + in_b) / probe["duplex_GBps"]) if duplex
                 else out_b / probe["d2h_GBps"] + in_b / probe["h2d_GBps"]) / 1e9
        dma["ideal_s"] = ideal
        dma["frac_of_measured_link"] = ideal / wall
        dma["duplex_overlap_measured"] = duplex
    plan_gpu_ms = sum(s["plan_gpu_ms"] for s in plan_stats) - sum(s["plan_gpu_ms"] for s in stats)
    nps = max(args.plan_steps, 1)
    host = [sum(s["plan_host_us"][i] for s in plan_stats) - sum(s["plan_host_us"][i] for s in stats)
            for i in range(3)]
    phases = [(sum(s["plan_phase_us"][i] for s in plan_stats) -
               sum(s["plan_phase_us"][i] for s in stats)) / nps for i in range(7)]
    floor_us = binding.probe_launch(100)
    plan = {"median": lat_dev["median"], "p99": lat_dev["p99"],
            "floor_us": floor_us,
            "floor": "one empty kernel launch, event record and wait (the plan is one launch "
                     "per pool; its lists come back through mapped host memory)",
            "c_call_median": lat_dev["c_call_median"], "c_call_p99": lat_dev["c_call_p99"],
            "inputs": "device memory (distances and masks already in HBM)",
            "host_inputs": dict(lat_host, inputs="host memory (numpy arrays; the call copies "
                                "them into pinned memory the plan kernel reads over the host "
                                "link)"),
            "core_phases_us": dict(zip(("classify", "cuts_sorts_prefixes", "demand_victims",
                                        "acceptance_setup", "acceptance", "lists",
                                        "publish"), phases)),
            "gpu_kernels_us": 1e3 * plan_gpu_ms / nps,
            "host_enqueue_us": host[0] / nps, "host_wait_us": host[1] / nps,
            "host_readback_us": host[2] / nps,
            "host_enqueue_parts_us": dict(zip(
                ("inputs", "stream_waits", "plan_launch", "other"),
                [(sum(s["plan_enqueue_us"][i] for s in plan_stats) -
                  sum(s["plan_enqueue_us"][i] for s in stats)) / nps for i in range(4)]))}

    rr = trace.pools[0] if args.workload == "roundrobin" else W.make_trace("roundrobin", 0).pools[0]
    loader = (None if args.no_loader else
              loader_bench(args, binding, W, rr, PoolMemory, DeviceBuffer, probe))
    objects = None if args.no_objects else object_bench(args, binding, W, DeviceBuffer)
    estimators = None if args.no_estimators else estimator_bench(args, binding, W, DeviceBuffer)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(trace, args.warmup, args.cpu_steps, args.cpu_agents, thr, budget,
                           args.cpu_seconds)

    rec = {
        "metric": "evict+prefetch GB/s per step (HBM and host-link % of peak); plan latency us/step",
        "value": moved / wall / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * wall / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "config": {"workload": f"{args.workload}: {WORKLOAD_TEXT[args.workload]}",
                   "seed": args.seed, "threshold": thr, "budget_units": budget,
                   "staging_bytes": args.staging_mib << 20, "ring_slots": args.ring,
                   "write_back": "none (clean evictions)" if args.clean_evict else "every eviction",
                   "direct_limit_bytes": int(args.direct_mib * (1 << 20)),
                   "caller_stream": "null stream" if args.null_stream else "own non-blocking stream",
                   "caller_wait": ("ss_sync blocks" if args.blocking_wait else
                                   "ss_sync polls (SS_FLAG_POLL_WAIT)"),
                   "host_copies": ("one per agent" if args.host_copies == 0 else
                                   f"{args.host_copies} shared round-robin"),
                   "bytes_out": out_b, "bytes_in": in_b},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "dma": dma,
        "plan_latency_us": plan,
        "kernels": kern,
        "direct": direct if args.direct_mib else None,
        "loader": loader,
        "object_distances": objects,
        "estimators": estimators,
        "probe": probe,
        "fill": ({"steps": fill_steps, "GBps": fill_b / fill_wall / 1e9,
                  "ms_per_step": 1e3 * fill_wall / fill_steps,
                  "note": "first steps on the empty pool (not in value)"} if fill_steps else None),
        "step_wall_ms": {"median": 1e3 * float(np.median(step_wall)),
                         "max": 1e3 * float(np.max(step_wall))},
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
