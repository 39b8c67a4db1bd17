"""Invariants I1-I7 on every step of every workload."""
import numpy as np
import pytest

import workloads as W
from oracle import OraclePool
from oracle.invariants import check_step, check_i7

S = W.SENTINEL


def run_checked(tr, pool_index, theta, budget, steps=None, i7=False):
    p = tr.pools[pool_index]
    pool = OraclePool(p.capacity_units, p.agent_units, p.unit_bytes)
    T = tr.n_steps if steps is None else steps
    moved = 0
    for t in range(T):
        before = pool.resident.copy()
        plan = pool.plan_step(tr.dist[t], tr.active[t], theta, budget)
        check_step(pool, plan, tr.dist[t], tr.active[t], theta, budget, before)
        if i7:
            check_i7(pool, tr.dist[t], tr.active[t], theta)
        moved += len(plan.loads)
    return moved


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("theta", [0, 1, 2, 8, S])
def test_tiny(seed, theta):
    tr = W.make_trace("tiny", seed)
    run_checked(tr, 0, theta, None, i7=(theta == S))
    run_checked(tr, 0, theta, 20)


@pytest.mark.parametrize("name,pool_index", [("roundrobin", 0), ("bursty", 0),
                                             ("zipf_lora", 0), ("zipf_lora", 1)])
@pytest.mark.parametrize("theta", [0, 4, S])
def test_mid_workloads(name, pool_index, theta):
    tr = W.make_trace(name, 0)
    uniform = bool((tr.pools[pool_index].agent_units == tr.pools[pool_index].agent_units[0]).all())
    i7 = (theta == S) and uniform and tr.pools[pool_index].capacity_units % int(
        tr.pools[pool_index].agent_units[0]) == 0
    assert run_checked(tr, pool_index, theta, None, i7=i7) > 0


def test_bursty_with_budget():
    tr = W.make_trace("bursty", 1)
    run_checked(tr, 0, S, 500)


@pytest.mark.slow
def test_diffusion():
    tr = W.make_trace("diffusion", 0)
    run_checked(tr, 0, S, None, steps=120)
