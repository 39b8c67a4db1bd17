"""Write-back elision (reading R13): with a dirty mask only changed victims
are written back; without one, every victim is (R9).  Bytes stay conserved:
a clean victim's host copy is already its content."""
import numpy as np
import pytest

import workloads as W
from oracle import OraclePool, BytePool, apply_step_bytes, run_trace

S = W.SENTINEL


def test_no_mask_writes_back_every_victim():
    tr = W.make_trace("roundrobin", 0)
    _, plans = run_trace(tr, S, steps=40)
    for p in plans:
        assert p.written.tolist() == p.victims.tolist()
        assert p.units_written == p.units_out and p.bytes_out == p.units_out * p.unit_bytes


def test_all_clean_writes_back_nothing_and_plans_are_unchanged():
    tr = W.make_trace("zipf_lora", 0)
    clean = np.zeros_like(tr.active)
    _, a = run_trace(tr, S, pool_index=1, steps=60)
    _, b = run_trace(tr, S, pool_index=1, steps=60, dirty=clean)
    for pa, pb in zip(a, b):
        assert pa.victims.tolist() == pb.victims.tolist()
        assert pa.loads.tolist() == pb.loads.tolist()
        assert pa.load_units.tolist() == pb.load_units.tolist()
        assert pb.bytes_out == 0 and len(pb.written) == 0
    assert sum(p.bytes_out for p in a) > 0


def test_mixed_mask_bytes_and_conservation():
    tr = W.shrink_planes(W.make_trace("tiny", 3), lambda p: [16, 32])
    p = tr.pools[0]
    rng = np.random.default_rng(0)
    dirty = (rng.random(tr.active.shape) < 0.5).astype(np.uint8)
    content = W.Content(p)
    host = {a: content.agent_bytes(a) for a in range(tr.n_agents)}
    frozen = {a: h.copy() for a, h in host.items()}
    pool = OraclePool(p.capacity_units, p.agent_units, p.unit_bytes)
    bp = BytePool(p.capacity_units, p.chunk_bytes)
    got_written = 0
    for t in range(tr.n_steps):
        plan = pool.plan_step(tr.dist[t], tr.active[t], S, None, dirty[t])
        exp = [int(v) for v in plan.victims if dirty[t][v]]
        assert plan.written.tolist() == exp
        assert plan.bytes_out == sum(int(p.agent_units[v]) for v in exp) * p.unit_bytes
        written = {}
        apply_step_bytes(bp, plan, p.agent_units, lambda a: host[a],
                         lambda a, b: written.__setitem__(a, b.copy()))
        assert sorted(written) == sorted(exp)
        for v, b in written.items():
            assert np.array_equal(b, frozen[v])
        got_written += len(exp)
        for a in np.flatnonzero(pool.resident):
            assert np.array_equal(bp.gather(pool.bt[a]), frozen[a])
    assert got_written > 0
