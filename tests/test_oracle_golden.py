"""Oracle against the paper's worked examples and the fixed readings.

Fixtures live in tests/golden/*.json, each with its citation; expectations
were derived by hand from the cited passage."""
import glob
import json
import os

import numpy as np
import pytest

from oracle import OraclePool, OvercommitError

FIX = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.json")))


def replay(fx, pool):
    N = len(fx["agent_units"])
    for t, st in enumerate(fx["steps"]):
        active = np.zeros(N, dtype=np.uint8)
        active[st["active"]] = 1
        exp = st["expect"]
        if "error" in exp:
            before = ([b.copy() for b in pool.bt], pool.resident.copy(), pool.owner.copy())
            with pytest.raises(OvercommitError):
                pool.plan_step(st["dist"], active, fx["threshold"], fx["budget"])
            assert all((a == b).all() for a, b in zip(before[0], pool.bt))
            assert (before[1] == pool.resident).all() and (before[2] == pool.owner).all()
            continue
        plan = pool.plan_step(st["dist"], active, fx["threshold"], fx["budget"])
        assert plan.victims.tolist() == exp["victims"], (t, plan.victims)
        assert plan.loads.tolist() == exp["loads"], (t, plan.loads)
        assert plan.n_demand == exp["n_demand"], t
        if "block_table" in exp:
            assert [b.tolist() for b in pool.bt] == exp["block_table"], t


@pytest.mark.parametrize("path", FIX, ids=[os.path.basename(p)[:-5] for p in FIX])
def test_fixture(path):
    fx = json.load(open(path))
    assert fx["cite"]
    replay(fx, OraclePool(fx["capacity_units"], fx["agent_units"]))


def test_fixtures_present():
    names = {os.path.basename(p)[:-5] for p in FIX}
    assert {"limitation_evict_farther", "optimized_timeline_prefetch", "prefetch_example"} <= names
