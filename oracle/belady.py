"""Independent references used to pin the oracle (parity pins, not policy).

TEST INFRASTRUCTURE: imported by the tests only.

* ``belady_min_loads``: Belady's MIN (Belady 1966) for requests that are sets
  of pages: on a miss, evict the resident pages not requested now whose next
  request lies farthest in the future.  It computes next-request times from
  the request sequence itself, never from a distance input.
* ``optimal_loads``: exhaustive dynamic programming over resident sets, the
  minimum number of loads any policy (demand or prefetching) can achieve.

With unit-size agents, a threshold of 0 (no prefetch) and exact distances,
the memory manager's eviction rule (largest distance first, only when memory
is insufficient) is exactly MIN, and MIN is optimal.
"""
from __future__ import annotations

from itertools import combinations


def belady_min_loads(requests, capacity: int) -> int:
    T = len(requests)
    resident: set = set()
    loads = 0
    for t, R in enumerate(requests):
        R = set(R)
        missing = R - resident
        loads += len(missing)
        overflow = len(resident) + len(missing) - capacity
        if overflow > 0:
            def next_request(a):
                for u in range(t + 1, T):
                    if a in requests[u]:
                        return u
                return T + 1                    # never again: farthest of all
            others = sorted(resident - R, key=next_request, reverse=True)
            for a in others[:overflow]:
                resident.discard(a)
        resident |= missing
    return loads


def optimal_loads(requests, n_items: int, capacity: int) -> int:
    """Minimum total loads over all resident-set sequences with
    ``R_t subset of S_t`` and ``|S_t| <= capacity``; cost of a transition is
    ``|S_t - S_{t-1}|``."""
    states = [frozenset(c) for k in range(capacity + 1)
              for c in combinations(range(n_items), k)]
    best = {frozenset(): 0}
    for R in requests:
        R = frozenset(R)
        nxt = {}
        for S in states:
            if not R <= S:
                continue
            nxt[S] = min(cost + len(S - P) for P, cost in best.items())
        best = nxt
    return min(best.values())
