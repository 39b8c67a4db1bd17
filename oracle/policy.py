"""Oracle of one simulation step of the invocation-distance memory manager.

TEST INFRASTRUCTURE.  This module is the plain, slow reference that the HIP
path is checked against.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does.

It follows the paper's method in the paper's order:

* invocation distance as a relative urgency (Section 3.2): only the order of
  distances matters, so every decision below compares keys
  ``(d, agent id)``;
* active agents have distance zero (Section 3.3, the prefetch example);
* reactive loading of an active agent whose memory is not on the GPU
  (Section 3.1, "Frequent reactive memory swaps"), with eviction only when
  memory is insufficient and largest distance first (Section 3.3,
  "Future reuse-aware eviction"; Appendix A, Table
  "agent-mem-interface", ``Evict(size, agentDistances)``);
* distance-guided prefetch of offloaded agents below a threshold, into free
  space or by replacing inactive residents of strictly larger distance
  (Section 3.3, "Distance-guided proactive prefetch"; Appendix A,
  ``DispatchLoadTasks(agentDistances, threshold, budget)``);
* one pool per memory module, every module planned with the same distances
  (Appendix A: modules register with the runtime independently).

Where the paper is silent the oracle takes these readings (each one is a
fixed rule that the HIP path must reproduce):

* R1  "smaller than that of any inactive resident" = smaller than at least
      one (the largest), because agent 4 is refused only for being larger
      than *all* inactive residents;
* R3  strict comparisons: ``D < threshold`` and victim ``d > d`` of the
      candidate it makes room for (no swap on a tie);
* R4  ties broken by agent id through ``key = d * 2**32 + id``: evict the
      larger key first, prefetch the smaller key first, demand loads by id;
* R5  the activation mask is authoritative: an active agent's distance is 0;
* R6  variable sizes: evict the shortest prefix that frees enough (leftover
      stays free); prefetch stops at the first candidate that cannot be
      placed;
* R7  ``budget`` caps the prefetched units per step, ``None`` = no cap;
* R8  an active set larger than the pool is an error and changes nothing;
* R10 units: units free before the step in ascending index, then the units
      released by this step's victims in eviction order, are handed to the
      loads in load order (demand loads first, then prefetches), logical
      unit j in order;
* R11 whole-agent granularity per pool;
* R13 write-back elision (optional ``dirty`` mask): an evicted agent whose
      memory did not change since it was loaded still has a current host
      copy, so its units are released without being written back; without a
      mask every eviction writes back (R9).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SENTINEL = 0xFFFFFFFF


class OvercommitError(ValueError):
    """The active agents alone need more units than the pool has (R8)."""


@dataclass
class Plan:
    victims: np.ndarray        # agent ids, eviction order (key descending)
    loads: np.ndarray          # agent ids, demand loads (id order) then prefetches (key ascending)
    n_demand: int              # leading entries of `loads` that are demand loads
    n_demand_victims: int      # leading entries of `victims` evicted for demand
    victim_units: np.ndarray   # physical units released by the eviction, victim then j order
    load_units: np.ndarray     # physical units written by the loads, load then j order
    units_out: int             # units released by the victims
    units_in: int
    unit_bytes: int
    written: np.ndarray = None       # victims whose bytes are written back, eviction order
    written_units: np.ndarray = None  # their units, victim then j order
    units_written: int = 0

    @property
    def bytes_out(self) -> int:
        return self.units_written * self.unit_bytes

    @property
    def bytes_in(self) -> int:
        return self.units_in * self.unit_bytes


class OraclePool:
    """State of one memory module's pool: which agents are resident and the
    block table ``bt[a][j]`` = physical unit of agent a's logical unit j."""

    def __init__(self, capacity_units: int, agent_units, unit_bytes: int = 1):
        self.U = int(capacity_units)
        self.s = np.asarray(agent_units, dtype=np.int64).copy()
        assert (self.s >= 1).all()
        self.N = len(self.s)
        self.unit_bytes = int(unit_bytes)
        self.resident = np.zeros(self.N, dtype=bool)
        self.bt = [np.full(int(k), -1, dtype=np.int64) for k in self.s]
        self.owner = np.full(self.U, -1, dtype=np.int64)   # agent owning each unit, -1 = free

    # ------------------------------------------------------------------
    def plan_step(self, D, active, threshold: int, budget=None, dirty=None) -> Plan:
        D = np.asarray(D, dtype=np.uint64)
        act = np.asarray(active).astype(bool)
        s, res, N = self.s, self.resident, self.N
        ids = np.arange(N, dtype=np.uint64)

        # 0. the active agents alone must fit (R8); nothing changes otherwise
        if int(s[act].sum()) > self.U:
            raise OvercommitError("active agents need %d units, pool has %d"
                                  % (int(s[act].sum()), self.U))

        # 1. distances and keys: active agents have distance 0 (R5, R4)
        d = np.where(act, np.uint64(0), D)
        key = (d << np.uint64(32)) | ids

        # 2. demand: active agents whose memory is not resident, by id;
        #    evict only what the free space cannot cover
        L = np.flatnonzero(act & ~res)
        free = self.U - int(s[res].sum())
        demand_units = int(s[L].sum())
        need = demand_units - free

        # 3. eviction order: inactive residents, largest key first
        E = np.flatnonzero(res & ~act)
        E = E[np.argsort(key[E], kind="stable")[::-1]]

        # 4. demand victims: shortest prefix of E that frees `need` units
        n_d, freed = 0, 0
        while freed < need:
            freed += int(s[E[n_d]])          # R8 guarantees E is long enough
            n_d += 1
        free_after_demand = free + freed - demand_units

        # 5. prefetch candidates: offloaded, inactive, below the threshold,
        #    smallest key first (R3, R4)
        C = np.flatnonzero(~res & ~act & (D < np.uint64(threshold)))
        C = C[np.argsort(key[C], kind="stable")]

        # 6-7. accept candidates in order while they fit into free space or
        #      into space of further inactive residents with strictly larger
        #      distance; stop at the first that does not (R1, R3, R6, R7)
        n_v, n_p = n_d, 0
        n, extra, S = n_d, 0, 0
        for i in range(len(C)):
            c = C[i]
            S += int(s[c])
            if budget is not None and S > budget:
                break
            while free_after_demand + extra < S and n < len(E):
                extra += int(s[E[n]])
                n += 1
            if free_after_demand + extra < S:
                break
            if n > n_d and d[E[n - 1]] <= d[c]:
                break
            n_p, n_v = i + 1, n

        V = E[:n_v]
        P = C[:n_p]
        loads = np.concatenate([L, P]).astype(np.int64)

        # 9. release the victims' units; remember which units were free before
        free_before = np.flatnonzero(self.owner < 0)
        released = []
        for v in V:
            released.append(self.bt[v].copy())
            self.owner[self.bt[v]] = -1
            self.bt[v][:] = -1
            self.resident[v] = False
        victim_units = (np.concatenate(released) if released
                        else np.zeros(0, dtype=np.int64))
        # R13: only victims whose memory changed are written back
        wmask = (np.ones(len(V), dtype=bool) if dirty is None
                 else np.asarray(dirty)[V].astype(bool))
        written = V[wmask]
        written_units = (np.concatenate([r for r, w in zip(released, wmask) if w])
                         if wmask.any() else np.zeros(0, dtype=np.int64))

        # 10. hand out units (R10): old free units ascending, then released ones
        F = np.concatenate([free_before, victim_units]).astype(np.int64)
        pos = 0
        load_units = []
        for a in loads:
            k = int(s[a])
            u = F[pos:pos + k]
            pos += k
            assert (self.owner[u] < 0).all()
            self.bt[a][:] = u
            self.owner[u] = a
            self.resident[a] = True
            load_units.append(u)
        load_units = (np.concatenate(load_units) if load_units
                      else np.zeros(0, dtype=np.int64))

        return Plan(victims=V.astype(np.int64), loads=loads, n_demand=len(L),
                    n_demand_victims=n_d, victim_units=victim_units,
                    load_units=load_units, units_out=int(s[V].sum()),
                    units_in=int(s[loads].sum()), unit_bytes=self.unit_bytes,
                    written=written.astype(np.int64), written_units=written_units,
                    units_written=int(s[written].sum()))

    # ------------------------------------------------------------------
    def block_table_csr(self):
        """(agent_off[N+1], units[sum s]) with -1 for non-resident agents."""
        off = np.concatenate([[0], np.cumsum(self.s)]).astype(np.int64)
        units = (np.concatenate(self.bt) if self.N else np.zeros(0, np.int64))
        return off, units


def run_trace(trace, threshold: int, budget=None, pool_index: int = 0, steps=None,
              use_true_distance: bool = False, on_step=None, dirty=None):
    """Replay a trace through one pool; returns the list of plans."""
    p = trace.pools[pool_index]
    pool = OraclePool(p.capacity_units, p.agent_units, p.unit_bytes)
    dist = trace.dist_true if use_true_distance else trace.dist
    T = trace.n_steps if steps is None else steps
    plans = []
    for t in range(T):
        plan = pool.plan_step(dist[t], trace.active[t], threshold, budget,
                              None if dirty is None else dirty[t])
        plans.append(plan)
        if on_step is not None:
            on_step(t, pool, plan)
    return pool, plans
