"""Object distances (Appendix A, fine-grained distance assignment)."""
import json
import os

import numpy as np

import workloads as W
from oracle.objects import object_distances

S = W.SENTINEL


def test_paper_example_min_of_sharers():
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "objects", "shared_object_min.json")))
    d, a = object_distances(fx["obj_off"], np.array(fx["obj_agents"]), np.array(fx["dist"]),
                            np.array(fx["active"]))
    assert d.tolist() == fx["expect_dist"] and a.tolist() == fx["expect_active"]


def test_properties_on_a_prefix_tree():
    rng = np.random.default_rng(4)
    off, agents, sizes = W.prefix_tree_objects(200, 3, 4, seed=1)
    M = len(off) - 1
    assert off[-1] == len(agents) and len(sizes) == M
    # the root is shared by everyone, every agent has a private leaf
    assert off[1] - off[0] == 200 and all(off[M - 200 + i + 1] - off[M - 200 + i] == 1
                                          for i in range(200))
    for _ in range(20):
        D = rng.integers(1, 50, size=200).astype(np.uint32)
        D[rng.random(200) < 0.1] = S
        act = (rng.random(200) < 0.05).astype(np.uint8)
        d, a = object_distances(off, agents, D, act)
        for o in range(M):
            refs = agents[off[o]:off[o + 1]]
            if a[o]:
                assert d[o] == 0 and act[refs].any()
            else:
                assert not act[refs].any()
                assert d[o] == D[refs].min() and (d[o] <= D[refs]).all()
        # the root's distance is the minimum over everyone (or 0 if anyone is active)
        assert d[0] == (0 if act.any() else D.min())


def test_unreferenced_object_has_no_future_use():
    d, a = object_distances([0, 0, 1], np.array([0], np.uint32), np.array([5], np.uint32),
                            np.array([0], np.uint8))
    assert d.tolist() == [S, 5] and a.tolist() == [0, 0]


def test_unknown_agent_ids_are_skipped():
    d, a = object_distances([0, 2, 3], np.array([7, 1, 9], np.uint32), np.array([3, 4], np.uint32),
                            np.array([0, 0], np.uint8))
    assert d.tolist() == [4, S] and a.tolist() == [0, 0]
