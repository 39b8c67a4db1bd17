"""Byte conservation (I4) on the oracle's byte mover.

After every step, every resident agent's units hold exactly that agent's
content, every evicted agent's staged bytes equal its content, and the host
copies never change (content is immutable, Section 3.3)."""
import numpy as np
import pytest

import workloads as W
from oracle import OraclePool, BytePool, apply_step_bytes

S = W.SENTINEL


def run_bytes(tr, pool_index, theta, steps):
    p = tr.pools[pool_index]
    content = W.Content(p, seed=0, pool_index=pool_index)
    host = {a: content.agent_bytes(a) for a in range(tr.n_agents)}
    frozen = {a: h.copy() for a, h in host.items()}
    pool = OraclePool(p.capacity_units, p.agent_units, p.unit_bytes)
    bp = BytePool(p.capacity_units, p.chunk_bytes)
    written = {}
    for t in range(steps):
        plan = pool.plan_step(tr.dist[t], tr.active[t], theta)
        out, inn = apply_step_bytes(bp, plan, p.agent_units, lambda a: host[a],
                                    lambda a, b: written.__setitem__(a, b.copy()))
        assert len(out) == plan.bytes_out and len(inn) == plan.bytes_in
        for v in plan.victims:
            assert np.array_equal(written.pop(int(v)), frozen[int(v)])
        for a in np.flatnonzero(pool.resident):
            got = bp.gather(pool.bt[a])
            assert np.array_equal(got, frozen[a]), (t, a)
    for a in range(tr.n_agents):
        assert np.array_equal(host[a], frozen[a])


@pytest.mark.parametrize("theta", [0, 3, S])
def test_tiny_bytes(theta):
    run_bytes(W.make_trace("tiny", 0), 0, theta, 100)


def test_roundrobin_small_planes_bytes():
    tr = W.shrink_planes(W.make_trace("roundrobin", 0), lambda p: [16] * 4)
    run_bytes(tr, 0, S, 40)


def test_zipf_lora_small_planes_bytes():
    tr = W.shrink_planes(W.make_trace("zipf_lora", 0),
                         lambda p: [16 * (1 + (c % 3)) for c in range(min(p.n_planes, 7))])
    run_bytes(tr, 1, S, 30)
