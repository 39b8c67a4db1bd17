"""Side-by-side replay of a trace through the HIP library and the CPU oracle.

Used by the GPU parity tests and by ``__graft_entry__.smoke``.  Each step
compares, exactly: victims (eviction order), loads (demand then prefetch),
counts, unit totals, the whole block table, the resident flags, the bytes
written back to every victim's host copy, and the bytes of resident units in
the device pool (all of them or a seeded sample)."""
from __future__ import annotations

import sys
import time

import numpy as np

import workloads as W
from oracle import OraclePool
from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer, PoolMemory

S = W.SENTINEL
POISON = 0xA5


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class DeviceTrace:
    """A trace's distances and masks resident in device memory; ``dist(t)``
    and ``active(t)`` are the device addresses of step t's arrays."""

    def __init__(self, trace, device=0):
        self.N = trace.n_agents
        d = np.ascontiguousarray(trace.dist, dtype=np.uint32)
        a = np.ascontiguousarray(trace.active, dtype=np.uint8)
        self.d = DeviceBuffer(d.nbytes, device)
        self.a = DeviceBuffer(a.nbytes, device)
        self.d.upload(d)
        self.a.upload(a)

    def dist(self, t):
        return self.d.ptr + 4 * self.N * t

    def active(self, t):
        return self.a.ptr + self.N * t

    def free(self):
        self.d.free()
        self.a.free()


def upload_trace(trace, device=0):
    return DeviceTrace(trace, device)


def fill_host(mem, content, spec, batch_bytes=256 << 20):
    """Every agent's host copy := its content (agent, unit, plane order)."""
    units = spec.agent_units.astype(np.int64)
    N = len(units)
    batch_units = max(1, batch_bytes // spec.unit_bytes)
    a0 = 0
    while a0 < N:
        a1 = a0
        tot = 0
        while a1 < N and (tot == 0 or tot + units[a1] <= batch_units):
            tot += units[a1]
            a1 += 1
        A = np.repeat(np.arange(a0, a1), units[a0:a1])
        J = np.concatenate([np.arange(k) for k in units[a0:a1]])
        data = content.units_bytes(A, J).reshape(-1)
        off = int(mem.host_off[a0])
        mem.host_np[off:off + len(data)] = data
        a0 = a1


def run_parity(trace, pool_index=0, theta=S, budget=None, steps=None, check_bytes=True,
               slot_units=8, ring_slots=2, sample_units=None, bt_every=1, seed=0, label="",
               dirty=None, device_inputs=None, direct_bytes=0, stream=0, before_plan=None,
               move_stream=None, sync_every=1, host_inputs=False, check_mirrors=False):
    """``device_inputs(t) -> (distances_ptr, active_ptr)`` replaces the uploaded
    trace on the HIP side (the oracle side always reads ``trace``).
    ``direct_bytes``: the pool's direct-transfer limit (0 = always staged).
    ``stream``: the caller's stream of every call; ``before_plan(t, stream)``
    may queue work there before step t's plan.  ``move_stream``: the caller's
    stream of ``evict_pack`` and ``prefetch_unpack`` if not ``stream``.
    ``sync_every``: the host waits for the pool only every that many steps
    (and after the last), so a step's plan and copies overlap the previous
    step's copies in between; plans are still compared every step, the block
    table, residency and bytes at the steps that wait.  At each of those, the
    host copy of every agent that is not resident must hold its content.
    ``host_inputs``: distances and masks (and the dirty mask) are passed as
    host arrays (pageable numpy memory) instead of device pointers.
    ``check_mirrors``: the plan's device lists are read back and compared
    each step too."""
    assert sync_every >= 1
    assert sync_every == 1 or dirty is None, "the dirty-mask checks write host copies each step"
    spec = trace.pools[pool_index]
    ub = spec.unit_bytes
    staging_bytes = 2 * ring_slots * slot_units * ub
    log(f"[parity] {label or trace.name} pool={spec.name} N={trace.n_agents} "
        f"U={spec.capacity_units} unit={ub}B planes={spec.n_planes} theta={theta} "
        f"budget={budget} slot_units={slot_units} ring={ring_slots} direct={direct_bytes}")
    mem = PoolMemory(spec, staging_bytes, ring_slots)
    content = W.Content(spec, seed=seed, pool_index=pool_index)
    if check_bytes:
        fill_host(mem, content, spec)
    pool = mem.make_pool(timing=True, direct_bytes=direct_bytes)
    opool = OraclePool(spec.capacity_units, spec.agent_units, ub)
    dev = upload_trace(trace) if device_inputs is None and not host_inputs else None
    if host_inputs:
        h_dist = np.ascontiguousarray(trace.dist, dtype=np.uint32)
        h_act = np.ascontiguousarray(trace.active, dtype=np.uint8)
    d_dirty = None
    if dirty is not None:
        dm = np.ascontiguousarray(dirty, dtype=np.uint8)
        if not host_inputs:
            d_dirty = DeviceBuffer(dm.nbytes)
            d_dirty.upload(dm)
    T = trace.n_steps if steps is None else steps
    rng = np.random.default_rng(seed + 99)
    units_i64 = spec.agent_units.astype(np.int64)
    moved = 0
    t0 = time.time()
    for t in range(T):
        if host_inputs:
            d_ptr, a_ptr = h_dist[t].ctypes.data, h_act[t].ctypes.data
        else:
            d_ptr, a_ptr = (dev.dist(t), dev.active(t)) if dev is not None else device_inputs(t)
        if before_plan is not None:
            before_plan(t, stream)
        if dirty is None:
            w_ptr = 0
        elif host_inputs:
            w_ptr = dm[t].ctypes.data
        else:
            w_ptr = d_dirty.ptr + trace.n_agents * t
        g = pool.plan_step(d_ptr, a_ptr, theta, budget, stream, w_ptr)
        o = opool.plan_step(trace.dist[t], trace.active[t], theta, budget,
                            None if dirty is None else dirty[t])
        assert g["units_written"] == o.units_written, (label, t)
        assert np.array_equal(g["victim_written"].astype(bool),
                              np.isin(o.victims, o.written)), (label, t)
        if check_bytes and dirty is not None:
            # a written-back victim's host copy must be rewritten by this step
            for v in o.written:
                mem.host_copy(int(v))[:] = POISON
        assert g["victims"].tolist() == o.victims.tolist(), (label, t, "victims")
        assert g["loads"].tolist() == o.loads.tolist(), (label, t, "loads")
        assert g["n_demand"] == o.n_demand, (label, t)
        assert g["n_demand_victims"] == o.n_demand_victims, (label, t)
        assert g["units_out"] == o.units_out and g["units_in"] == o.units_in, (label, t)
        assert g["bytes_out"] == o.bytes_out and g["bytes_in"] == o.bytes_in, (label, t)
        if check_mirrors:
            # the plan's device lists, read on the plan's stream after the call
            nv, nl = len(o.victims), len(o.loads)
            dv = np.empty(max(nv, 1), np.uint32)
            dl = np.empty(max(nl, 1), np.uint32)
            B.stream_sync(stream)
            if nv:
                B.copy(dv.ctypes.data, g["d_victims"], 4 * nv)
            if nl:
                B.copy(dl.ctypes.data, g["d_loads"], 4 * nl)
            assert dv[:nv].tolist() == o.victims.tolist(), (label, t, "device victims")
            assert dl[:nl].tolist() == o.loads.tolist(), (label, t, "device loads")
        ms = stream if move_stream is None else move_stream
        pool.evict_pack(ms)
        pool.prefetch_unpack(ms)
        moved += o.units_in + o.units_out
        if t % sync_every != 0 and t != T - 1:
            continue
        pool.sync()
        if t % bt_every == 0 or t == T - 1:
            bt = pool.block_table_host_all()
            obt = np.concatenate(opool.bt)
            assert np.array_equal(bt, obt.astype(np.int32)), (label, t, "block table")
            assert np.array_equal(pool.resident_host().astype(bool), opool.resident), (label, t)
        if check_bytes:
            for v in o.victims:           # written back, or clean and still current
                v = int(v)
                exp = content.units_bytes(np.full(units_i64[v], v), np.arange(units_i64[v]))
                assert np.array_equal(mem.host_copy(v), exp.reshape(-1)), (label, t, "host", v)
            res = np.flatnonzero(opool.resident)
            if len(res):
                A = np.repeat(res, units_i64[res])
                J = np.concatenate([np.arange(units_i64[a]) for a in res])
                U = np.concatenate([opool.bt[a] for a in res])
                if sample_units is not None and len(U) > sample_units:
                    pick = rng.choice(len(U), sample_units, replace=False)
                    A, J, U = A[pick], J[pick], U[pick]
                got = mem.units_bytes(U)
                exp = content.units_bytes(A, J)
                bad = np.flatnonzero((got != exp).any(axis=1))
                assert len(bad) == 0, (label, t, "device bytes", A[bad[:4]], J[bad[:4]])
            if sync_every > 1:
                # steps since the last wait wrote back victims the host never
                # saw: every agent that is not resident now must have its
                # content in its host copy (its initial copy, or the bytes
                # written back when it was last evicted after a poisoning)
                off = np.flatnonzero(~opool.resident)
                if sample_units is not None and len(off) > sample_units:
                    off = rng.choice(off, sample_units, replace=False)
                for a in off:
                    a = int(a)
                    exp = content.units_bytes(np.full(units_i64[a], a), np.arange(units_i64[a]))
                    assert np.array_equal(mem.host_copy(a), exp.reshape(-1)), \
                        (label, t, "host copy of an offloaded agent", a)
            if dirty is None:
                for a in o.loads:         # a resident agent's host copy is stale by design
                    mem.host_copy(int(a))[:] = POISON
    st = pool.stats()
    pool.close()
    if dev is not None:
        dev.free()
    mem.free()
    if d_dirty is not None:
        d_dirty.free()
    log(f"[parity] {label or trace.name}: {T} steps ok, {moved} units moved, "
        f"{time.time() - t0:.1f}s")
    return st


def synthetic_trace(n_agents, capacity_units, n_steps, k_active, seed, units=None,
                    chunk_bytes=(32, 16), noisy=False):
    """A uniform random activation trace for edge cases."""
    rng = np.random.default_rng(seed)
    active = np.zeros((n_steps, n_agents), dtype=np.uint8)
    for t in range(n_steps):
        k = int(k_active(t, rng)) if callable(k_active) else int(k_active)
        if k:
            active[t, rng.choice(n_agents, k, replace=False)] = 1
    if units is None:
        units = np.ones(n_agents, dtype=np.uint32)
    pool = W.PoolSpec("syn", capacity_units, list(chunk_bytes), np.asarray(units, np.uint32))
    dt = W.exact_distances(active)
    dist = W.noisy_distances(dt, 2.0, rng) if noisy else dt.copy()
    return W.Trace(f"syn{n_agents}", n_agents, n_steps, [pool], active, dist, dt, {})
