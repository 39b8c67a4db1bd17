"""Failure handling through the C ABI: a HIP failure while moving data
poisons the pool (or the load scheduler), every later call reports
SS_ERR_POISONED, and destruction stays clean.

The failure is forced from the host with ``ss_debug_fail_copy``: the armed
copy command is refused before it is issued, so no kernel faults and the
device stays healthy (a fresh pool afterwards must work)."""
import numpy as np
import pytest

import workloads as W
from gpu_harness import fill_host, log, run_parity, upload_trace
from oracle import OraclePool
from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer, PoolMemory

pytestmark = pytest.mark.gpu
S = W.SENTINEL


@pytest.fixture(autouse=True)
def _disarm():
    assert B.device_count() > 0, "GPU tests need a GPU"
    B.debug_fail_copy(0)
    yield
    B.debug_fail_copy(0)


def _status(fn, *a):
    try:
        fn(*a)
    except B.ScaleSimError as e:
        return e.status
    return B.SS_OK


def _pool_after_good_steps(n_good):
    tr = W.make_trace("tiny", 0)
    spec = tr.pools[0]
    mem = PoolMemory(spec, 2 * 2 * 3 * spec.unit_bytes, 2)
    pool = mem.make_pool()                   # staged copies only (no direct transfers)
    dev = upload_trace(tr)
    opool = OraclePool(spec.capacity_units, spec.agent_units, spec.unit_bytes)
    t = 0
    for t in range(n_good):
        pool.plan_step(dev.dist(t), dev.active(t), S)
        opool.plan_step(tr.dist[t], tr.active[t], S)
        pool.evict_pack(0)
        pool.prefetch_unpack(0)
    pool.sync()
    return tr, mem, pool, dev, opool, n_good


def _next_step_with_moves(tr, pool, dev, opool, t):
    """Plan steps until one writes back and loads bytes; returns its index."""
    while True:
        g = pool.plan_step(dev.dist(t), dev.active(t), S)
        o = opool.plan_step(tr.dist[t], tr.active[t], S)
        assert g["victims"].tolist() == o.victims.tolist()
        if g["bytes_out"] > 0 and g["bytes_in"] > 0:
            return t, g
        pool.evict_pack(0)
        pool.prefetch_unpack(0)
        t += 1


def _assert_poisoned(pool, dev, t):
    P = B.SS_ERR_POISONED
    assert _status(pool.plan_step, dev.dist(t), dev.active(t), S) == P
    assert _status(pool.evict_pack, 0) == P
    assert _status(pool.prefetch_unpack, 0) == P
    assert _status(pool.sync) == P
    assert _status(pool.block_table_host_all) == P
    assert _status(pool.resident_host) == P
    assert "poisoned" in B.load().ss_last_error().decode()


def _fresh_pool_works():
    # the device is unharmed: a new pool replays the tiny workload exactly
    run_parity(W.make_trace("tiny", 1), theta=S, steps=15, slot_units=3, ring_slots=2,
               label="after failure")


@pytest.mark.parametrize("which", [1, 2])
def test_eviction_copy_failure_poisons_pool(which):
    tr, mem, pool, dev, opool, t = _pool_after_good_steps(12)
    try:
        t, g = _next_step_with_moves(tr, pool, dev, opool, t)
        log(f"[failure] evict step {t}: bytes_out {g['bytes_out']}, copy #{which} fails")
        n_copies = g["n_victims"]            # at least one copy per written-back victim
        B.debug_fail_copy(min(which, n_copies))
        assert _status(pool.evict_pack, 0) == B.SS_ERR_HIP
        assert "copy" in B.load().ss_last_error().decode() or \
            "unknown" in B.load().ss_last_error().decode()
        _assert_poisoned(pool, dev, t + 1)
    finally:
        B.debug_fail_copy(0)
        pool.close()                         # waits for the queued work, frees
        dev.free()
        mem.free()
    _fresh_pool_works()


def test_load_copy_failure_poisons_pool():
    tr, mem, pool, dev, opool, t = _pool_after_good_steps(12)
    try:
        t, g = _next_step_with_moves(tr, pool, dev, opool, t)
        pool.evict_pack(0)                   # every device-to-host copy issued normally
        log(f"[failure] load step {t}: bytes_in {g['bytes_in']}, first copy fails")
        B.debug_fail_copy(1)
        assert _status(pool.prefetch_unpack, 0) == B.SS_ERR_HIP
        _assert_poisoned(pool, dev, t + 1)
    finally:
        B.debug_fail_copy(0)
        pool.close()
        dev.free()
        mem.free()
    _fresh_pool_works()


def test_disarmed_hook_changes_nothing():
    B.debug_fail_copy(5)
    B.debug_fail_copy(0)
    _fresh_pool_works()


def test_loader_copy_failure_poisons_loader():
    tr = W.make_trace("tiny", 0)
    spec = tr.pools[0]
    mem = PoolMemory(spec, 2 * spec.unit_bytes, 2)          # one unit per slot
    fill_host(mem, W.Content(spec, seed=0), spec)
    units = np.arange(spec.capacity_units, dtype=np.int32)
    d_units = DeviceBuffer(units.nbytes)
    d_units.upload(units)
    L = B.Loader([mem.desc_args()])
    try:
        s = spec.agent_units.astype(np.int64)
        off = np.concatenate([[0], np.cumsum(s)])
        L.submit([(0, a, 10 + a, d_units.ptr + 4 * int(off[a])) for a in range(4)])
        assert len(L.pump(3)) == 3
        B.debug_fail_copy(2)                 # the second chunk from here fails
        st = _status(L.pump, 10)
        assert st == B.SS_ERR_HIP
        assert _status(L.pump, 1) == B.SS_ERR_POISONED
        assert _status(L.submit, [(0, 9, 1, d_units.ptr)]) == B.SS_ERR_POISONED
        L.sync()                             # the chunks issued before still land
    finally:
        B.debug_fail_copy(0)
        L.close()
        d_units.free()
        mem.free()
    _fresh_pool_works()
