"""Per-step invariants of the memory manager, checked on the oracle.

TEST INFRASTRUCTURE: imported by the tests only.

I1  no active agent is evicted;
I2  every active agent is resident after the step;
I3  the pool never overflows, and block table and unit owners agree;
I5  nothing is evicted and loaded in the same step;
I6  every prefetched agent is below the threshold, every victim taken to
    make room for a prefetch has strictly larger distance than that
    prefetch, and the prefetched units respect the budget;
I7  with unit sizes all equal (pool a whole number of agents), no budget and
    a threshold above every finite distance, a full pool after the step keeps
    no inactive resident farther than an offloaded candidate.
"""
from __future__ import annotations

import numpy as np

SENTINEL = 0xFFFFFFFF


def check_step(pool, plan, D, active, threshold, budget, resident_before):
    act = np.asarray(active).astype(bool)
    D = np.asarray(D, dtype=np.uint64)
    s = pool.s
    V = set(int(v) for v in plan.victims)
    Ld = set(int(a) for a in plan.loads)
    d = np.where(act, 0, D)

    assert not (V & set(np.flatnonzero(act).tolist())), "I1: active agent evicted"
    assert pool.resident[act].all(), "I2: active agent not resident"
    assert int(s[pool.resident].sum()) <= pool.U, "I3: pool overflow"
    units_seen = np.full(pool.U, -1, dtype=np.int64)
    for a in range(pool.N):
        bt = pool.bt[a]
        if pool.resident[a]:
            assert (bt >= 0).all() and (bt < pool.U).all(), "I3: bad unit"
            assert (units_seen[bt] < 0).all(), "I3: unit with two owners"
            units_seen[bt] = a
        else:
            assert (bt == -1).all(), "I3: stale block-table entry"
    assert (units_seen == pool.owner).all(), "I3: owner map disagrees with block table"
    assert not (V & Ld), "I5: agent evicted and loaded in one step"
    assert all(resident_before[v] for v in V), "victim was not resident"
    assert not any(resident_before[a] for a in Ld), "load of a resident agent"

    P = [int(a) for a in plan.loads[plan.n_demand:]]
    for p in P:
        assert int(D[p]) < threshold and not act[p], "I6: prefetch above threshold"
    if budget is not None:
        assert int(s[P].sum()) <= budget, "I6: budget exceeded"
    # pair prefetch victims with the prefetch they made room for
    free_before = pool.U - int(s[resident_before].sum())
    demand_units = int(s[plan.loads[:plan.n_demand]].sum())
    avail = free_before + int(s[plan.victims[:plan.n_demand_victims]].sum()) - demand_units
    assert avail >= 0
    e = plan.n_demand_victims
    for p in P:
        avail -= int(s[p])
        while avail < 0:
            v = int(plan.victims[e])
            assert int(d[v]) > int(d[p]), "I6: prefetch replaced a nearer agent"
            avail += int(s[v])
            e += 1
    assert e == len(plan.victims), "I6: victims beyond what the loads need"
    assert set(int(v) for v in plan.written) <= V, "written-back agent is not a victim"
    assert plan.units_written == int(s[plan.written].sum())


def check_i7(pool, D, active, threshold):
    """I7 (call only for equal sizes, no budget, threshold > all finite D)."""
    act = np.asarray(active).astype(bool)
    D = np.asarray(D, dtype=np.uint64)
    s0 = int(pool.s[0])
    free = pool.U - int(pool.s[pool.resident].sum())
    if free >= s0:
        return
    inact_res = pool.resident & ~act
    cand = ~pool.resident & ~act & (D < np.uint64(threshold))
    if inact_res.any() and cand.any():
        assert D[inact_res].max() <= D[cand].min(), "I7: farther agent kept over a nearer one"
