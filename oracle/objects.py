"""Oracle of fine-grained distance assignment for shared memory objects.

TEST INFRASTRUCTURE: imported by the tests and the smoke check only.

Appendix A, "Fine-grained distance assignment": a memory object referenced by
several agents (for example a node of a shared prefix tree) gets the minimum
invocation distance of the agents that currently reference it.  Reading R14:
the object is needed now if any referencing agent is active, and an active
object's distance is 0 (the activation mask is authoritative, R5); an object
that no agent references has no future use (distance 0xFFFFFFFF).  A
reference to an id outside the agent arrays names no agent and is skipped.
"""
from __future__ import annotations

import numpy as np

SENTINEL = 0xFFFFFFFF


def object_distances(obj_off, obj_agents, D, active):
    obj_off = np.asarray(obj_off, dtype=np.int64)
    M = len(obj_off) - 1
    dist = np.full(M, SENTINEL, dtype=np.uint32)
    act = np.zeros(M, dtype=np.uint8)
    for o in range(M):
        refs = [int(a) for a in obj_agents[obj_off[o]:obj_off[o + 1]] if int(a) < len(D)]
        if len(refs) == 0:
            continue
        if any(active[a] for a in refs):
            act[o] = 1
            dist[o] = 0
        else:
            dist[o] = min(int(D[a]) for a in refs)
    return dist, act
