"""HIP path against the CPU oracle, bit for bit, through the C ABI.

Every comparison is exact (tolerance 0): all of the path is integer indexing
and byte movement.  Cases:
  * the tiny workload at full size, seeds 0-4, thresholds 0 / 2 / none;
  * all five workloads at their full agent counts and pool capacities, every
    step, with the chunk sizes shrunk so that every agent's host copy fits
    (the plan does not depend on chunk sizes; bytes are still checked for
    every resident unit);
  * the real unit layouts (64 x 32 KiB KV pages, 448-plane LoRA adapters,
    512 KiB unified units) on agent subsets, with sampled byte checks;
  * every workload but the tiny one in the benchmark's own launch
    configuration (full size, real unit layouts, 1 GiB slots, shared host
    copies, no host wait between steps), plans every step, block tables every
    tenth step and bytes on sampled units;
  * distances and masks from host memory, and the plan's device lists;
  * the plan on one stream and the moves on another without host waits, so
    that a step's plan overlaps the previous step's copies;
  * direct transfers (a direction at or below the pool's direct_bytes moves
    by kernel straight between units and host copies): every step direct,
    and a limit that sends some steps' directions direct and others staged;
  * edge cases: one-unit ring slots, no prefetch, budgets, an agent count
    that is not a multiple of the wave or block size, lists larger than the
    plan kernel's LDS sort buffer, 2^20 agents, empty steps, overcommit and
    call order."""
import numpy as np
import pytest

import workloads as W
from gpu_harness import run_parity, synthetic_trace, upload_trace, log
from oracle import OraclePool, OvercommitError
from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer, PoolMemory

pytestmark = pytest.mark.gpu
S = W.SENTINEL


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert B.device_count() > 0, "GPU tests need a GPU"


def small(trace, planes=(32, 48)):
    return W.shrink_planes(trace, lambda p: list(planes))


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("theta", [0, 2, S])
def test_tiny_full_size(seed, theta):
    run_parity(W.make_trace("tiny", seed), theta=theta, slot_units=3, ring_slots=2,
               label=f"tiny s{seed} t{theta}")


def test_tiny_one_unit_slots():
    st = run_parity(W.make_trace("tiny", 1), theta=S, slot_units=1, ring_slots=1,
                    label="tiny one-unit ring")
    assert st["pack_launches"] > 100 and st["unpack_launches"] > 100


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("theta", [0, S])
def test_tiny_direct(seed, theta):
    st = run_parity(W.make_trace("tiny", seed), theta=theta, slot_units=3, ring_slots=2,
                    direct_bytes=1 << 40, label=f"tiny direct s{seed} t{theta}")
    assert st["pack_launches"] == 0 and st["unpack_launches"] == 0
    # steps that both write back and load move both directions in one launch
    assert st["duplex_launches"] > 50
    assert st["direct_out_launches"] + st["duplex_launches"] > 50
    assert st["direct_in_launches"] + st["duplex_launches"] > 50
    assert st["d2h_bytes"] == 0 and st["h2d_bytes"] == 0


@pytest.mark.parametrize("name,n_agents,steps,pool_index,limit_units", [
    ("bursty", 150, 40, 0, 24),        # 64 x 32 KiB units, lognormal agent sizes
    ("zipf_lora", 40, 40, 0, 64),      # KV pool, 32-unit agents
    ("zipf_lora", 40, 40, 1, 2),       # 448-plane LoRA slots
    ("diffusion", 150, 40, 0, 300),    # 512 KiB unified units
])
def test_direct_and_staged_mixed(name, n_agents, steps, pool_index, limit_units):
    """A limit between small and large steps: each direction of each step
    goes direct or staged on its own, so both orders of the eviction/load
    hazard (direct pack then staged unpack and the reverse) occur."""
    tr = W.subsample_agents(W.make_trace(name, 0), n_agents)
    spec = tr.pools[pool_index]
    slot_units = max(1, (64 << 20) // spec.unit_bytes)
    st = run_parity(tr, pool_index=pool_index, theta=S, steps=steps, slot_units=slot_units,
                    ring_slots=2, sample_units=48, direct_bytes=limit_units * spec.unit_bytes,
                    label=f"{name}[{pool_index}] direct<={limit_units}u")
    assert st["direct_out_launches"] + st["duplex_launches"] > 0
    assert st["direct_in_launches"] + st["duplex_launches"] > 0
    assert st["pack_launches"] > 0 and st["unpack_launches"] > 0


@pytest.mark.parametrize("case", range(6))
def test_random_pipeline_shapes(case):
    """Seeded random ring sizes, slot sizes and direct-transfer limits on a
    variable-size workload: every ordering of copies, packs and unpacks the
    pipeline can produce (ring reuse, the release hazard, the wait for the
    next pack, direct and staged directions mixed) against the oracle."""
    rng = np.random.default_rng(1000 + case)
    tr = W.subsample_agents(W.make_trace("bursty", case % 3), 120)
    tr = W.shrink_planes(tr, lambda p: [32, 16])
    ring = int(rng.choice([1, 2, 3, 5]))
    slot_units = int(rng.integers(1, 40))
    direct = int(rng.choice([0, 0, 8, 64])) * tr.pools[0].unit_bytes
    run_parity(tr, theta=S, steps=60, slot_units=slot_units, ring_slots=ring, direct_bytes=direct,
               label=f"random shape {case}: ring {ring}, slot {slot_units}u, direct {direct}B")


@pytest.mark.parametrize("name,pool_index", [("roundrobin", 0), ("bursty", 0), ("zipf_lora", 0),
                                             ("zipf_lora", 1), ("diffusion", 0)])
def test_workload_full_counts(name, pool_index):
    tr = small(W.make_trace(name, 0))
    sample = 20000 if name == "diffusion" else None
    run_parity(tr, pool_index=pool_index, theta=S, slot_units=4096, ring_slots=2,
               sample_units=sample, label=f"{name}[{pool_index}] full counts")


@pytest.mark.parametrize("name,steps,watched", [("roundrobin", None, 0), ("zipf_lora", None, 0),
                                                ("bursty", 150, 0), ("diffusion", 60, 64)])
def test_bench_configuration_sampled(name, steps, watched):
    # A workload as bench.py times it: full size, real unit layouts (2 MiB
    # units of 64 x 32 KiB; for the LoRA workload also 80 MiB adapter slots of
    # 448 planes in a second pool planned with the same inputs; 512 KiB units
    # in one 160 GB pool for the 50,000-agent workload), 8 GiB of staging per
    # pool in four slots per direction, a 4 MiB direct limit, 128 host copies
    # per pool shared round-robin by the agents, a stream of the caller's own
    # and the pools' polled waits; the host waits for the pool only every
    # tenth step.  Plans match the
    # oracle at every step; block tables and residency every tenth step and
    # after the last.  Bytes are checked where one step fixes them, on sampled
    # units every tenth step: a victim whose host copy no other agent moving
    # in the step shares must leave its device bytes there, and such a load
    # must receive the bytes its host copy held before the step.  Where a step
    # moves so many agents that every shared copy has several movers (the
    # 50,000-agent workload), `watched` sampled agents get private host copies.
    tr = W.make_trace(name, 0)
    if steps is not None:
        tr = W.Trace(tr.name, tr.n_agents, steps, tr.pools, tr.active[:steps], tr.dist[:steps],
                     tr.dist_true[:steps], tr.meta)
    n_host = 128
    slot_of = np.arange(tr.n_agents, dtype=np.int64) % n_host
    if watched:
        watch = np.random.default_rng(5).choice(tr.n_agents, watched, replace=False)
        slot_of[watch] = n_host + np.arange(watched)
    n_slots = int(slot_of.max()) + 1
    ctx = []
    for pi, spec in enumerate(tr.pools):
        ub = spec.unit_bytes
        mem = PoolMemory(spec, 8192 << 20, 4, host_slots=slot_of)
        words = int(spec.agent_units.max()) * ub // 8
        pattern = np.arange(words, dtype=np.uint64)
        host64 = mem.host_np.view(np.uint64)
        for k in range(n_slots):  # every 8-byte word of both pools' host copies distinct
            host64[k * words:(k + 1) * words] = pattern + np.uint64((pi << 56) | ((k + 1) << 40))
        del pattern, host64
        units = spec.agent_units.astype(np.int64)
        ctx.append(dict(spec=spec, ub=ub, mem=mem, units=units,
                        row=np.concatenate([[0], np.cumsum(units)]),
                        pool=mem.make_pool(timing=True, direct_bytes=4 << 20, poll_wait=True),
                        opool=OraclePool(spec.capacity_units, spec.agent_units, ub)))
    dev = upload_trace(tr)
    stream = B.Stream()
    rng = np.random.default_rng(7)
    checked_v = checked_l = 0

    def unique_movers(group, movers):
        counts = np.bincount(slot_of[np.asarray(movers, dtype=np.int64)], minlength=n_slots)
        return [int(a) for a in group if counts[slot_of[int(a)]] == 1]

    def sample_units(units, a):
        return sorted({0, int(units[a]) // 2, int(units[a]) - 1})

    def read_units(mem, phys):
        # the sampled units' chunks only (whole-plane reads would move GBs)
        out = np.empty((len(phys), mem.spec.unit_bytes), dtype=np.uint8)
        off = 0
        for c, cb in enumerate(mem.spec.chunk_bytes):
            for k, u in enumerate(phys):
                out[k, off:off + cb] = mem.planes[c].download(int(u) * cb, cb)
            off += cb
        return out

    try:
        for t in range(tr.n_steps):
            check = t % 10 == 5
            if check:
                for c in ctx:
                    c["pool"].sync()
                    c["bt_before"] = c["pool"].block_table_host_all().copy()
            for c in ctx:
                g = c["pool"].plan_step(dev.dist(t), dev.active(t), S, None, stream.handle)
                o = c["opool"].plan_step(tr.dist[t], tr.active[t], S)
                assert g["victims"].tolist() == o.victims.tolist(), (name, t)
                assert g["loads"].tolist() == o.loads.tolist(), (name, t)
                assert g["bytes_out"] == o.bytes_out and g["bytes_in"] == o.bytes_in, (name, t)
                c["v_before"], c["l_before"] = {}, {}
                if check:
                    movers = np.concatenate([o.victims, o.loads])
                    vs = unique_movers(o.victims, movers)
                    ls = unique_movers(o.loads, movers)
                    for v in [vs[i] for i in rng.permutation(len(vs))[:2]]:
                        js = sample_units(c["units"], v)
                        rows = c["bt_before"][c["row"][v] + np.asarray(js)]
                        assert (rows >= 0).all(), (name, t, v)
                        c["v_before"][v] = (js, read_units(c["mem"], rows))
                    for a in [ls[i] for i in rng.permutation(len(ls))[:2]]:
                        js = sample_units(c["units"], a)
                        hc = c["mem"].host_copy(a).reshape(-1, c["ub"])
                        c["l_before"][a] = (js, hc[js].copy())
            for c in ctx:
                c["pool"].evict_pack(stream.handle)
            for c in ctx:
                c["pool"].prefetch_unpack(stream.handle)
            if check:
                for c in ctx:
                    pool, mem, ub = c["pool"], c["mem"], c["ub"]
                    pool.sync()
                    bt = pool.block_table_host_all()
                    assert np.array_equal(bt, np.concatenate(c["opool"].bt).astype(np.int32)), \
                        (name, t)
                    assert np.array_equal(pool.resident_host().astype(bool),
                                          c["opool"].resident), (name, t)
                    for v, (js, exp) in c["v_before"].items():
                        got = mem.host_copy(v).reshape(-1, ub)[js]
                        assert np.array_equal(got, exp), (name, t, "victim host copy", v)
                        checked_v += len(js)
                    for a, (js, exp) in c["l_before"].items():
                        got = read_units(mem, bt[c["row"][a] + np.asarray(js)])
                        assert np.array_equal(got, exp), (name, t, "loaded units", a)
                        checked_l += len(js)
        for c in ctx:
            c["pool"].sync()
            assert np.array_equal(c["pool"].block_table_host_all(),
                                  np.concatenate(c["opool"].bt).astype(np.int32)), name
        log(f"[bench config] {name}: {tr.n_steps} steps, {checked_v} victim and {checked_l} "
            f"load units checked")
        assert checked_v > 0 and checked_l > 0
    finally:
        stream.sync()
        stream.close()
        for c in ctx:
            c["pool"].close()
            c["mem"].free()
        dev.free()


@pytest.mark.parametrize("name,theta,budget", [("roundrobin", 0, None), ("bursty", 0, None),
                                               ("bursty", S, 500), ("roundrobin", 4, 300),
                                               ("diffusion", 3, None)])
def test_workload_thresholds_and_budgets(name, theta, budget):
    tr = small(W.make_trace(name, 1), planes=(16,))
    steps = 150 if name == "diffusion" else None
    run_parity(tr, theta=theta, budget=budget, steps=steps, slot_units=2048, ring_slots=3,
               sample_units=5000, label=f"{name} t{theta} b{budget}")


@pytest.mark.parametrize("name,n_agents,steps,pool_index", [
    ("roundrobin", 40, 60, 0),     # 64 planes x 32 KiB
    ("bursty", 150, 40, 0),        # same unit, lognormal sizes
    ("zipf_lora", 40, 60, 1),      # 448 planes of 32-448 KiB, 80 MiB units
    ("diffusion", 150, 40, 0),     # one 512 KiB plane
])
def test_real_layouts(name, n_agents, steps, pool_index):
    tr = W.subsample_agents(W.make_trace(name, 0), n_agents)
    spec = tr.pools[pool_index]
    slot_units = max(1, (256 << 20) // spec.unit_bytes)
    run_parity(tr, pool_index=pool_index, theta=S, steps=steps, slot_units=slot_units,
               ring_slots=3, sample_units=48, label=f"{name} layout sub{n_agents}")


@pytest.mark.parametrize("mode", ["clean", "mixed"])
def test_write_back_elision(mode):
    tr = W.make_trace("tiny", 4)
    rng = np.random.default_rng(11)
    dirty = (np.zeros(tr.active.shape, np.uint8) if mode == "clean"
             else (rng.random(tr.active.shape) < 0.4).astype(np.uint8))
    st = run_parity(tr, theta=S, slot_units=2, ring_slots=2, dirty=dirty, label=f"elision {mode}")
    if mode == "clean":
        assert st["pack_launches"] == 0 and st["d2h_bytes"] == 0
    trb = W.shrink_planes(W.make_trace("bursty", 2), lambda p: [32, 16])
    dirty = (rng.random(trb.active.shape) < (0.0 if mode == "clean" else 0.5)).astype(np.uint8)
    run_parity(trb, theta=S, slot_units=512, ring_slots=3, dirty=dirty, steps=120,
               label=f"bursty elision {mode}")


@pytest.mark.parametrize("mode", ["clean", "mixed"])
def test_write_back_elision_direct(mode):
    """Write-back elision with direct transfers: only the dirty victims'
    units are gathered into their host copies (the per-unit host offsets
    cover written-back victims only)."""
    tr = W.make_trace("tiny", 3)
    rng = np.random.default_rng(12)
    dirty = (np.zeros(tr.active.shape, np.uint8) if mode == "clean"
             else (rng.random(tr.active.shape) < 0.4).astype(np.uint8))
    st = run_parity(tr, theta=S, slot_units=2, ring_slots=2, dirty=dirty, direct_bytes=1 << 40,
                    label=f"direct elision {mode}")
    assert st["pack_launches"] == 0 and st["unpack_launches"] == 0
    if mode == "clean":
        # nothing is written back: loads alone, never the two-way launch
        assert st["direct_out_launches"] == 0 and st["direct_out_bytes"] == 0
        assert st["duplex_launches"] == 0
    else:
        # clean victims' released units are loaded without a write-back
        assert st["direct_out_launches"] + st["duplex_launches"] > 0


def test_two_pools_share_streams():
    """The KV and LoRA pools of one workload stepped together (they share the
    device's streams), each against its own oracle, bytes included."""
    from oracle import OraclePool
    tr = W.shrink_planes(W.make_trace("zipf_lora", 1), lambda p: [32, 16, 48][:2 + p.n_planes % 2])
    dev = upload_trace(tr)
    mems, pools, opools, contents = [], [], [], []
    for k, spec in enumerate(tr.pools):
        mem = PoolMemory(spec, 2 * 2 * 64 * spec.unit_bytes, 2)
        c = W.Content(spec, seed=0, pool_index=k)
        from gpu_harness import fill_host
        fill_host(mem, c, spec)
        mems.append(mem)
        contents.append(c)
        pools.append(mem.make_pool())
        opools.append(OraclePool(spec.capacity_units, spec.agent_units, spec.unit_bytes))
    for t in range(tr.n_steps):
        plans = [p.plan_step(dev.dist(t), dev.active(t), S) for p in pools]
        for p in pools:
            p.evict_pack(0)
        for p in pools:
            p.prefetch_unpack(0)
        for k, (p, op) in enumerate(zip(pools, opools)):
            o = op.plan_step(tr.dist[t], tr.active[t], S)
            assert plans[k]["victims"].tolist() == o.victims.tolist(), (k, t)
            assert plans[k]["loads"].tolist() == o.loads.tolist(), (k, t)
        for p in pools:
            p.sync()
        for k, (p, op, mem, c) in enumerate(zip(pools, opools, mems, contents)):
            assert np.array_equal(p.block_table_host_all(), np.concatenate(op.bt).astype(np.int32))
            res = np.flatnonzero(op.resident)
            s = tr.pools[k].agent_units.astype(np.int64)
            A = np.repeat(res, s[res])
            J = np.concatenate([np.arange(s[a]) for a in res])
            U = np.concatenate([op.bt[a] for a in res])
            assert np.array_equal(mem.units_bytes(U), c.units_bytes(A, J)), (k, t)
            for a in plans[k]["loads"]:
                mem.host_copy(int(a))[:] = 0xA5
    for p in pools:
        p.close()
    for m in mems:
        m.free()
    dev.free()


def test_ragged_agent_count_and_sizes():
    rng = np.random.default_rng(5)
    units = rng.integers(1, 9, size=1037).astype(np.uint32)
    tr = synthetic_trace(1037, 900, 60, lambda t, r: r.integers(0, 60), seed=5, units=units,
                         noisy=True)
    run_parity(tr, theta=S, slot_units=37, ring_slots=2, label="ragged 1037")
    run_parity(tr, theta=5, budget=40, slot_units=37, ring_slots=2, label="ragged 1037 t5 b40")


def test_lists_beyond_lds_sort_buffer():
    # 40,000 unit-size agents, room for 20,000: the evictable list and the
    # candidate prefix both exceed the 16,384 keys the plan kernel sorts in LDS
    tr = synthetic_trace(40000, 20000, 25, 600, seed=11, chunk_bytes=(16,))
    run_parity(tr, theta=S, slot_units=8192, ring_slots=2, sample_units=4000,
               label="global sort path")


def test_cut_sets_beyond_lds():
    # 40,000 unit-size agents, room for 20,000.  Step 0 fills the pool with
    # agents that never run again; at step 1 the other 20,000 agents are one
    # step away, so the plan swaps the whole pool: the evictable residents it
    # must sort (20,000) and the candidates it may accept (20,000) both exceed
    # the plan kernel's 16,384-key LDS buffer and take the global-memory sorts.
    n, cap = 40000, 20000
    active = np.zeros((4, n), np.uint8)
    active[0, :cap] = 1
    active[2, cap:] = 1
    dist = W.exact_distances(active)
    pool = W.PoolSpec("syn", cap, [16], np.ones(n, np.uint32))
    tr = W.Trace("swap40000", n, 4, [pool], active, dist, dist.copy(), {})
    run_parity(tr, theta=S, slot_units=8192, ring_slots=2, sample_units=4000,
               label="cut sets beyond LDS")


@pytest.mark.parametrize("n,cap", [(8000, 4000), (8292, 4100), (16000, 8000)])
def test_joint_sort_sizes(n, cap):
    # Step 0 fills the pool with agents that never run again; at step 1, 100
    # other agents run (demand loads) and the rest (at most cap of them, so
    # that step 2 fits) are one step away (candidates), so the plan sorts the
    # whole pool (T = cap keys), the 100 demand loads and n - cap - 100
    # candidates.  Their union takes the plan core's joint LDS sort up to 8,192
    # keys (8,000: padded to 8,192) and the separate sorts beyond (8,192 + 100;
    # 16,000).
    active = np.zeros((4, n), np.uint8)
    active[0, :cap] = 1
    active[1, cap:cap + 100] = 1
    active[2, cap + 100:] = 1
    dist = W.exact_distances(active)
    pool = W.PoolSpec("syn", cap, [16], np.ones(n, np.uint32))
    tr = W.Trace(f"joint{n}", n, 4, [pool], active, dist, dist.copy(), {})
    run_parity(tr, theta=S, slot_units=8192, ring_slots=2, sample_units=4000,
               label=f"joint sort {n} agents")


@pytest.mark.parametrize("capacity", [65536, 65600, 524320])
def test_free_unit_scan_pool_sizes(capacity):
    # The plan picks the pre-step free units from the occupancy bitmap with
    # each thread holding ceil(words / 1024) words: up to 2 in registers (pools
    # up to 65,536 units), up to 16 (524,288 units), a loop beyond.  2,000
    # agents of about capacity / 600 units each, 30 of them run per step, so
    # every step evicts and the free units left by earlier steps are reused.
    rng = np.random.default_rng(capacity)
    per = capacity // 600
    units = rng.integers(per // 2, per + per // 2, size=2000).astype(np.uint32)
    tr = synthetic_trace(2000, capacity, 10, 30, seed=capacity, units=units, chunk_bytes=(16,),
                         noisy=True)
    run_parity(tr, theta=S, slot_units=65536, ring_slots=2, sample_units=4000,
               label=f"free-unit scan, {capacity} units")


@pytest.mark.parametrize("n_agents", [40000, 50000])
@pytest.mark.parametrize("theta,budget", [(S, None), (3, None), (S, 300)])
def test_many_agents_variable_sizes(n_agents, theta, budget):
    # the multi-workgroup plan path with ragged sizes, noisy distances, a
    # pool of about a tenth of all units and several hundred activations per
    # step: candidate cuts, evictable cuts, thresholds and budgets
    rng = np.random.default_rng(n_agents)
    units = rng.integers(1, 9, size=n_agents).astype(np.uint32)
    cap = int(units.sum()) // 10
    tr = synthetic_trace(n_agents, cap, 24, lambda t, r: r.integers(200, 600), seed=n_agents,
                         units=units, chunk_bytes=(16,), noisy=True)
    run_parity(tr, theta=theta, budget=budget, slot_units=8192, ring_slots=2, sample_units=3000,
               label=f"{n_agents} agents t{theta} b{budget}")


@pytest.mark.parametrize("theta,budget", [(S, None), (3, 5000)])
def test_million_agents(theta, budget):
    # The largest agent count of the tests: 2^20 one-unit agents (20 id bits,
    # 256 classifying workgroups) sharing a 65,536-unit pool, 30,000 of them
    # active per step with noisy distances, so that steps evict and load
    # 20,000-38,000 agents: evictable and candidate sets far beyond the plan
    # kernel's LDS sorts (its global-memory sorts), budgets and thresholds.
    tr = synthetic_trace(1 << 20, 65536, 6, 30000, seed=21, chunk_bytes=(16,), noisy=True)
    run_parity(tr, theta=theta, budget=budget, slot_units=65536, ring_slots=2, sample_units=4000,
               label=f"2^20 agents t{theta} b{budget}")


@pytest.mark.parametrize("direct", [0, 1 << 20])
def test_block_table_tail_many_items(direct):
    # 1,190-1,790 victims and 1,190-4,400 loads per step among 12,001 agents
    # (the fused plan core's limit is 12,288): more than the 16 waves x 64
    # items that its block-table tail takes in one batch, so every wave runs
    # more than one batch.
    rng = np.random.default_rng(31)
    n = 12001
    units = rng.integers(1, 3, size=n).astype(np.uint32)
    tr = synthetic_trace(n, 9000, 8, 4400, seed=31, units=units, chunk_bytes=(16,))
    run_parity(tr, theta=0, slot_units=1024, ring_slots=2, direct_bytes=direct,
               label=f"tail batches, direct={direct}")


@pytest.mark.parametrize("n_agents", [4097, 12288, 12289])
def test_classification_batch_edges(n_agents):
    # agent counts around the plan's one-workgroup limit (12,288) and one past
    # a 4,096-agent classification batch, with ragged sizes and noisy distances
    rng = np.random.default_rng(n_agents)
    units = rng.integers(1, 4, size=n_agents).astype(np.uint32)
    tr = synthetic_trace(n_agents, n_agents // 3, 20, n_agents // 50, seed=n_agents, units=units,
                         chunk_bytes=(16,), noisy=True)
    run_parity(tr, theta=S, slot_units=2048, ring_slots=2, sample_units=3000,
               label=f"classification edges {n_agents}")


def test_plan_queued_behind_long_work():
    # Work queued on the caller's stream before a plan holds its kernel back
    # for longer than the host polls the plan's flag (2 ms), so the call falls
    # back to the plan's event; the plans must match the oracle either way.
    n = 50_000
    rng = np.random.default_rng(21)
    pos = np.ascontiguousarray(rng.integers(0, 4096, size=(n, 2)).astype(np.int32))
    p = DeviceBuffer(pos.nbytes)
    p.upload(pos)
    d = DeviceBuffer(4 * n)
    d.upload(rng.integers(0, 1000, size=n).astype(np.uint32))
    out = DeviceBuffer(4 * n)
    wsb = B.interaction_distances_workspace(n)
    ws = DeviceBuffer(max(wsb, 4))
    s = B.Stream()

    def busy(t, stream):
        if t % 3 == 0:                       # about 16 x 0.2 ms of kernels
            for _ in range(16):
                B.interaction_distances(p.ptr, d.ptr, n, 3, 2, out.ptr, ws.ptr, wsb, stream)

    try:
        tr = synthetic_trace(600, 250, 12, 40, seed=21, chunk_bytes=(16,))
        run_parity(tr, theta=S, slot_units=64, ring_slots=2, stream=s.handle,
                   before_plan=busy, label="plan behind long work")
    finally:
        s.sync()
        s.close()
        for b in (p, d, out, ws):
            b.free()


@pytest.mark.parametrize("direct", [0, 1 << 20])
def test_moves_on_another_stream_than_the_plan(direct):
    # The plan runs on one caller stream (behind kernels queued there every
    # other step) and the step's moves on another: the packs and unpacks must
    # still follow the plan's block-table update, queued on the plan's stream.
    n = 50_000
    rng = np.random.default_rng(23)
    pos = np.ascontiguousarray(rng.integers(0, 4096, size=(n, 2)).astype(np.int32))
    p = DeviceBuffer(pos.nbytes)
    p.upload(pos)
    d = DeviceBuffer(4 * n)
    d.upload(rng.integers(0, 1000, size=n).astype(np.uint32))
    out = DeviceBuffer(4 * n)
    wsb = B.interaction_distances_workspace(n)
    ws = DeviceBuffer(max(wsb, 4))
    s_plan, s_move = B.Stream(), B.Stream()

    def busy(t, stream):
        if t % 2 == 0:
            for _ in range(4):
                B.interaction_distances(p.ptr, d.ptr, n, 3, 2, out.ptr, ws.ptr, wsb, stream)

    try:
        tr = synthetic_trace(300, 120, 12, 25, seed=23, chunk_bytes=(16,))
        run_parity(tr, theta=S, slot_units=32, ring_slots=2, stream=s_plan.handle,
                   move_stream=s_move.handle, before_plan=busy, direct_bytes=direct,
                   sync_every=3, label=f"moves on another stream, direct={direct}")
    finally:
        s_plan.sync()
        s_move.sync()
        s_plan.close()
        s_move.close()
        for b in (p, d, out, ws):
            b.free()


def test_empty_steps_and_idle_pool():
    tr = synthetic_trace(100, 40, 30, lambda t, r: 0 if t % 3 else r.integers(0, 30), seed=2)
    run_parity(tr, theta=S, slot_units=5, ring_slots=2, label="empty steps")


def test_sentinel_and_extreme_distances():
    tr = synthetic_trace(300, 120, 40, 20, seed=3, chunk_bytes=(16,))
    d = tr.dist.copy()
    rng = np.random.default_rng(3)
    d[rng.random(d.shape) < 0.2] = S
    d[rng.random(d.shape) < 0.1] = S - 1
    tr.dist[:] = d
    for theta in (S, S - 1, 1):
        run_parity(tr, theta=theta, slot_units=64, ring_slots=2, label=f"extreme t{theta}")


def test_overcommit_and_call_order():
    units = np.full(8, 3, dtype=np.uint32)
    tr = synthetic_trace(8, 9, 3, 0, seed=0, units=units)
    tr.active[0, [0, 1]] = 1
    tr.active[1, [0, 1, 2, 3]] = 1        # 12 units > 9: overcommit
    tr.active[2, [2]] = 1
    spec = tr.pools[0]
    mem = PoolMemory(spec, 2 * 2 * spec.unit_bytes * 3, 2)
    pool = mem.make_pool()
    dev = upload_trace(tr)
    st = 0
    with pytest.raises(B.ScaleSimError) as e:
        pool.evict_pack(st)
    assert e.value.status == B.SS_ERR_ORDER
    p0 = pool.plan_step(dev.dist(0), dev.active(0), S, None, st)
    assert p0["loads"].tolist() == [0, 1]
    with pytest.raises(B.ScaleSimError) as e:
        pool.plan_step(dev.dist(0), dev.active(0), S, None, st)
    assert e.value.status == B.SS_ERR_ORDER
    with pytest.raises(B.ScaleSimError) as e:
        pool.prefetch_unpack(st)
    assert e.value.status == B.SS_ERR_ORDER
    pool.evict_pack(st)
    pool.prefetch_unpack(st)
    bt_before = pool.block_table_host_all().copy()
    res_before = pool.resident_host().copy()
    with pytest.raises(B.OvercommitError):
        pool.plan_step(dev.dist(1), dev.active(1), S, None, st)
    assert np.array_equal(pool.block_table_host_all(), bt_before)
    assert np.array_equal(pool.resident_host(), res_before)
    p2 = pool.plan_step(dev.dist(2), dev.active(2), S, None, st)
    assert p2["n_demand"] == 1 and p2["loads"][0] == 2
    pool.evict_pack(st)
    pool.prefetch_unpack(st)
    pool.sync()
    pool.close()
    dev.free()
    mem.free()


@pytest.mark.parametrize("n_agents", [64, 12289])
def test_overcommit_between_streams(n_agents):
    # Overcommitted steps between good ones, each step's calls on another
    # caller stream, with the plan core classifying the agents itself (64)
    # and after the multi-workgroup classification (12,289, where the
    # block-table update runs as kernels that must see the overcommit and
    # change nothing): plans, block table and residency match the oracle.
    cap = 40 if n_agents < 100 else 100
    # active agents per step (unit-size agents): over capacity at steps 1 and
    # 3, exactly at capacity at step 5
    counts = [cap * 6 // 10, cap * 13 // 10, cap * 4 // 10, cap + 1, cap * 7 // 10, cap, cap // 2]
    tr = synthetic_trace(n_agents, cap, len(counts), lambda t, r: counts[t], seed=n_agents,
                         chunk_bytes=(16,))
    spec = tr.pools[0]
    mem = PoolMemory(spec, 2 * 2 * 16 * spec.unit_bytes, 2)
    pool = mem.make_pool()
    opool = OraclePool(spec.capacity_units, spec.agent_units, spec.unit_bytes)
    dev = upload_trace(tr)
    streams = [B.Stream(), B.Stream()]
    try:
        for t in range(tr.n_steps):
            st = streams[t % 2].handle
            log(f"[overcommit] N={n_agents} step {t} active={counts[t]}")
            if counts[t] > spec.capacity_units:
                with pytest.raises(B.OvercommitError):
                    pool.plan_step(dev.dist(t), dev.active(t), S, None, st)
                with pytest.raises(OvercommitError):
                    opool.plan_step(tr.dist[t], tr.active[t], S)
            else:
                g = pool.plan_step(dev.dist(t), dev.active(t), S, None, st)
                o = opool.plan_step(tr.dist[t], tr.active[t], S)
                assert g["victims"].tolist() == o.victims.tolist(), (n_agents, t)
                assert g["loads"].tolist() == o.loads.tolist(), (n_agents, t)
                pool.evict_pack(st)
                pool.prefetch_unpack(st)
            pool.sync()
            obt = np.concatenate(opool.bt).astype(np.int32)
            assert np.array_equal(pool.block_table_host_all(), obt), (n_agents, t)
            assert np.array_equal(pool.resident_host().astype(bool), opool.resident), (n_agents, t)
    finally:
        for s_ in streams:
            s_.sync()
            s_.close()
        pool.close()
        dev.free()
        mem.free()


@pytest.mark.parametrize("name", ["tiny", "roundrobin", "diffusion"])
def test_host_inputs(name):
    # Distances and masks passed as host arrays (pageable numpy memory): the
    # call copies them into pinned memory that the plan kernel reads over the
    # host link.  One workgroup plans the 64- and 1,000-agent workloads, the
    # classification over many workgroups the 50,000-agent one.  The plan's
    # device lists are compared with the oracle every step too.
    if name == "tiny":
        tr, slot, sample, steps = W.make_trace("tiny", 0), 3, None, None
    else:
        tr, slot = small(W.make_trace(name, 0)), 4096
        sample, steps = (20000, 120) if name == "diffusion" else (None, None)
    run_parity(tr, theta=S, steps=steps, slot_units=slot, ring_slots=2, sample_units=sample,
               host_inputs=True, check_mirrors=True, label=f"{name} host inputs")


def test_mixed_host_and_device_inputs():
    # host distances with a device mask, on the multi-workgroup plan path
    tr = synthetic_trace(12289, 4000, 12, 150, seed=41, chunk_bytes=(16,), noisy=True)
    dev = upload_trace(tr)
    h_dist = np.ascontiguousarray(tr.dist, dtype=np.uint32)
    try:
        run_parity(tr, theta=S, slot_units=1024, ring_slots=2, sample_units=2000,
                   device_inputs=lambda t: (h_dist[t].ctypes.data, dev.active(t)),
                   check_mirrors=True, label="host distances, device mask")
    finally:
        dev.free()


def test_write_back_elision_host_mask():
    tr = W.make_trace("tiny", 2)
    rng = np.random.default_rng(13)
    dirty = (rng.random(tr.active.shape) < 0.4).astype(np.uint8)
    run_parity(tr, theta=S, slot_units=2, ring_slots=2, dirty=dirty, host_inputs=True,
               label="elision, host mask")


def test_short_device_input_is_rejected():
    # a device pointer with fewer than N elements left in its allocation is
    # refused before any work, and the pool is unchanged
    tr = synthetic_trace(16, 8, 2, 2, seed=0)
    spec = tr.pools[0]
    mem = PoolMemory(spec, 4 * spec.unit_bytes, 1)
    pool = mem.make_pool()
    dev = upload_trace(tr)
    try:
        last = dev.d.ptr + dev.d.nbytes - 4 * 15          # 15 of 16 elements left
        with pytest.raises(B.ScaleSimError) as e:
            pool.plan_step(last, dev.active(0), S)
        assert e.value.status == B.SS_ERR_ARG
        g = pool.plan_step(dev.dist(0), dev.active(0), S)
        o = OraclePool(spec.capacity_units, spec.agent_units).plan_step(tr.dist[0], tr.active[0], S)
        assert g["loads"].tolist() == o.loads.tolist()
        pool.evict_pack(0)
        pool.prefetch_unpack(0)
        pool.sync()
    finally:
        pool.close()
        dev.free()
        mem.free()


@pytest.mark.parametrize("direct", [0, 1 << 20])
def test_plan_and_moves_on_two_streams_without_waits(direct):
    # Ordering between a step's evictions and the next step's plan: the plan
    # runs on one caller stream, the moves on another, and the host waits for
    # the pool only every eighth step.  Many small ring slots keep a step's
    # packs and device-to-host copies running while the next plan is queued;
    # that plan's block-table update rewrites the lists those packs read, its
    # unpacks may overwrite units the packs have not read yet, and its
    # host-to-device copies may read host copies still being written, unless
    # the plan waits for the evictions.  Block table, residency, resident bytes
    # and the host copy of every offloaded agent are compared at each wait.
    tr = W.shrink_planes(W.make_trace("bursty", 0), lambda p: [2048, 2048])
    s_plan, s_move = B.Stream(), B.Stream()
    try:
        run_parity(tr, theta=S, steps=120, slot_units=48, ring_slots=2, sample_units=3000,
                   stream=s_plan.handle, move_stream=s_move.handle, sync_every=8,
                   direct_bytes=direct, label=f"two streams, no waits, direct={direct}")
    finally:
        s_plan.sync()
        s_move.sync()
        s_plan.close()
        s_move.close()
