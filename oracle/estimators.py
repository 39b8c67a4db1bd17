"""Oracle of the on-device invocation-distance estimators.

TEST INFRASTRUCTURE: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg only.

Section 3.2 defines the distance per kind of simulation:

* predefined activation paths: an agent's distance is its hop count from the
  origin of the propagation along the network (breadth-first activation);
* interaction-involved simulations: D = min(D_action, D_interaction), where
  D_interaction is the physical distance to another agent divided by the
  movement velocity.

Readings where the text leaves room (each reproduced by the HIP path):

* R17 hop counts: a multi-source breadth-first search along the graph's
  directed edges (u -> v: u passes information to v) from the given sources
  (the agents holding the information now, hop 0); a vertex reached first
  after k edges has distance k; vertices not reached within ``max_hops``
  edges (or never) have no predicted activation (0xFFFFFFFF).  Source ids
  outside the graph are skipped; repeated sources are one source.
* R18 interaction: positions on an integer tile grid, Euclidean distance to
  the nearest other agent, a conversation radius r (tiles) and a closing
  speed v (tiles per step, >= 1), so D_interaction = floor(max(0, dist - r)
  / v) steps; with integer r and v this equals
  floor(max(0, isqrt(d2) - r) / v) for the squared distance d2, so the whole
  computation is exact in integers.  An agent with no other agent has no
  interaction term (0xFFFFFFFF).
"""
from __future__ import annotations

import math
from collections import deque

import numpy as np

SENTINEL = 0xFFFFFFFF


def hop_distances(row_off, col, sources, max_hops=None):
    """Breadth-first hop counts from ``sources`` over the CSR graph
    (``col[row_off[u]:row_off[u+1]]`` are u's out-neighbours)."""
    V = len(row_off) - 1
    hops = np.full(V, SENTINEL, dtype=np.uint32)
    q = deque()
    for s in sources:
        s = int(s)
        if 0 <= s < V and hops[s] == SENTINEL:
            hops[s] = 0
            q.append(s)
    while q:
        u = q.popleft()
        h = int(hops[u])
        if max_hops is not None and h >= max_hops:
            continue
        for v in col[int(row_off[u]):int(row_off[u + 1])]:
            v = int(v)
            if 0 <= v < V and hops[v] == SENTINEL:
                hops[v] = h + 1
                q.append(v)
    return hops


def interaction_distance_one(pos, i, d_action_i, velocity, radius=0):
    """D of agent i: min(D_action, D_interaction) over all other agents."""
    assert velocity >= 1 and radius >= 0
    best = None
    xi, yi = int(pos[i][0]), int(pos[i][1])
    for j in range(len(pos)):
        if j == i:
            continue
        dx = xi - int(pos[j][0])
        dy = yi - int(pos[j][1])
        d2 = dx * dx + dy * dy
        if best is None or d2 < best:
            best = d2
    if best is None:
        return int(d_action_i)
    return min(int(d_action_i), max(0, math.isqrt(best) - radius) // velocity)


def interaction_distances(pos, d_action, velocity, radius=0):
    """D = min(D_action, D_interaction) per agent; ``pos`` is int [N, 2]."""
    pos = np.asarray(pos, dtype=np.int64).tolist()
    d_action = np.asarray(d_action, dtype=np.uint32)
    return np.array([interaction_distance_one(pos, i, d_action[i], velocity, radius)
                     for i in range(len(pos))], dtype=np.uint32)
