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


# ---------------------------------------------------------------------------
# The checker must fire: each corruption below breaks one invariant and must
# raise that invariant's own assertion.
# ---------------------------------------------------------------------------

import copy


def _prefetch_step(theta=S):
    """A tiny-workload step (after the pool filled) whose plan prefetches
    at least one agent by evicting one; returns the state needed by
    check_step, with the step already applied to the pool."""
    tr = W.make_trace("tiny", 0)
    p = tr.pools[0]
    pool = OraclePool(p.capacity_units, p.agent_units, p.unit_bytes)
    for t in range(tr.n_steps):
        before = pool.resident.copy()
        plan = pool.plan_step(tr.dist[t], tr.active[t], theta, None)
        if t > 10 and len(plan.loads) > plan.n_demand and \
                len(plan.victims) > plan.n_demand_victims:
            check_step(pool, plan, tr.dist[t], tr.active[t], theta, None, before)
            return pool, plan, tr.dist[t].copy(), tr.active[t].copy(), before
    raise AssertionError("no prefetching step")


def test_checker_passes_the_uncorrupted_step():
    pool, plan, D, act, before = _prefetch_step()
    check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_an_evicted_active_agent():
    pool, plan, D, act, before = _prefetch_step()
    bad = copy.copy(plan)
    bad.victims = np.concatenate([plan.victims, [np.flatnonzero(act)[0]]])
    with pytest.raises(AssertionError, match="I1"):
        check_step(pool, bad, D, act, S, None, before)


def test_checker_flags_an_active_agent_left_offloaded():
    pool, plan, D, act, before = _prefetch_step()
    a = int(np.flatnonzero(act)[0])
    pool.resident[a] = False
    with pytest.raises(AssertionError, match="I2"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_an_overflow():
    pool, plan, D, act, before = _prefetch_step()
    pool.resident[:] = True                  # every agent resident: far over capacity
    with pytest.raises(AssertionError, match="I3: pool overflow"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_a_unit_with_two_owners():
    pool, plan, D, act, before = _prefetch_step()
    a, b = [int(x) for x in np.flatnonzero(pool.resident)[:2]]
    pool.bt[b] = pool.bt[a].copy()
    with pytest.raises(AssertionError, match="I3: unit with two owners"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_a_stale_block_table_row():
    pool, plan, D, act, before = _prefetch_step()
    a = int(np.flatnonzero(~pool.resident)[0])
    pool.bt[a][0] = 0
    with pytest.raises(AssertionError, match="I3: stale block-table entry"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_an_owner_map_mismatch():
    pool, plan, D, act, before = _prefetch_step()
    u = int(pool.bt[int(np.flatnonzero(pool.resident)[0])][0])
    pool.owner[u] = -1
    with pytest.raises(AssertionError, match="I3: owner map"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_an_agent_evicted_and_loaded():
    pool, plan, D, act, before = _prefetch_step()
    bad = copy.copy(plan)
    bad.loads = np.concatenate([plan.loads, plan.victims[:1]])
    with pytest.raises(AssertionError, match="I5"):
        check_step(pool, bad, D, act, S, None, before)


def test_checker_flags_a_prefetch_above_the_threshold():
    pool, plan, D, act, before = _prefetch_step()
    P = plan.loads[plan.n_demand:]
    theta = int(D[P].max())                  # the farthest prefetch is not below this
    with pytest.raises(AssertionError, match="I6: prefetch above threshold"):
        check_step(pool, plan, D, act, theta, None, before)


def test_checker_flags_a_budget_overrun():
    pool, plan, D, act, before = _prefetch_step()
    P = plan.loads[plan.n_demand:]
    budget = int(pool.s[P].sum()) - 1
    with pytest.raises(AssertionError, match="I6: budget exceeded"):
        check_step(pool, plan, D, act, S, budget, before)


def test_checker_flags_a_prefetch_that_replaced_a_nearer_agent():
    pool, plan, D, act, before = _prefetch_step()
    # every prefetch victim now as near as the last prefetch: no longer
    # strictly farther than the prefetch it made room for
    P = plan.loads[plan.n_demand:]
    Vp = plan.victims[plan.n_demand_victims:]
    D = D.copy()
    D[Vp] = D[P].max()
    with pytest.raises(AssertionError, match="I6: prefetch replaced a nearer agent"):
        check_step(pool, plan, D, act, S, None, before)


def test_checker_flags_victims_beyond_need():
    pool, plan, D, act, before = _prefetch_step()
    victims = set(plan.victims.tolist())
    extra = [int(a) for a in np.flatnonzero(before & ~act) if a not in victims]
    bad = copy.copy(plan)
    bad.victims = np.concatenate([plan.victims, extra[:1]])
    with pytest.raises(AssertionError, match="I6: victims beyond what the loads need"):
        check_step(pool, bad, D, act, S, None, before)


def test_i7_flags_a_farther_resident_kept_over_a_nearer_candidate():
    # a full pool of unit-size agents: resident 0 (inactive, distance 9)
    # while offloaded agent 2 (distance 1) is a candidate
    pool = OraclePool(2, np.ones(4, np.int64), 1)
    pool.resident[[0, 1]] = True
    pool.bt[0][:] = 0
    pool.bt[1][:] = 1
    pool.owner[:] = [0, 1]
    D = np.array([9, 3, 1, 5], np.uint32)
    act = np.array([0, 1, 0, 0], np.uint8)
    with pytest.raises(AssertionError, match="I7"):
        check_i7(pool, D, act, S)
    D[0] = 1                                 # now no farther than the nearest candidate
    check_i7(pool, D, act, S)
