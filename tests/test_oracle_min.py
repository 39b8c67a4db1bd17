"""Textbook reduction and brute force.

With unit-size agents, no prefetch (threshold 0) and exact distances, the
eviction rule (largest distance first, only when memory is insufficient;
Section 3.3 'Future reuse-aware eviction') is Belady's MIN for set requests,
so total loads must equal an independently written MIN simulator, and MIN
must equal the exhaustive optimum.  With prefetch on, loads can only be
higher than that optimum."""
import numpy as np
import pytest

import workloads as W
from oracle import run_trace
from oracle.belady import belady_min_loads, optimal_loads

S = W.SENTINEL


def total_loads(plans):
    return sum(len(p.loads) for p in plans)


def requests_of(trace):
    return [set(np.flatnonzero(trace.active[t]).tolist()) for t in range(trace.n_steps)]


@pytest.mark.parametrize("seed", range(5))
def test_tiny_workload_equals_min(seed):
    tr = W.make_trace("tiny", seed)
    p = tr.pools[0]
    _, plans = run_trace(tr, threshold=0, use_true_distance=True)
    cap = p.capacity_units // int(p.agent_units[0])
    assert total_loads(plans) == belady_min_loads(requests_of(tr), cap)


@pytest.mark.parametrize("pool_index", [0, 1])
def test_zipf_lora_pools_equal_min(pool_index):
    tr = W.make_trace("zipf_lora", 0)
    p = tr.pools[pool_index]
    assert (p.agent_units == p.agent_units[0]).all()
    _, plans = run_trace(tr, threshold=0, pool_index=pool_index, use_true_distance=True)
    cap = p.capacity_units // int(p.agent_units[0])
    assert total_loads(plans) == belady_min_loads(requests_of(tr), cap)


def test_random_tiny_traces_min_dp_oracle():
    rng = np.random.default_rng(1234)
    n_checked = 0
    for it in range(120):
        n = int(rng.integers(3, 8))
        cap = int(rng.integers(1, min(4, n - 1) + 1))
        k_act = int(rng.integers(1, cap + 1))
        T = int(rng.integers(4, 13))
        tr = W.random_tiny_trace(rng, n, T, k_act, cap)
        reqs = requests_of(tr)
        opt = optimal_loads(reqs, n, cap)
        assert belady_min_loads(reqs, cap) == opt
        _, plans = run_trace(tr, threshold=0, use_true_distance=True)
        assert total_loads(plans) == opt, it
        for theta in (1, 2, S):
            _, plans = run_trace(tr, threshold=theta, use_true_distance=True)
            assert total_loads(plans) >= opt
        n_checked += 1
    assert n_checked == 120


def test_min_detects_wrong_eviction_order():
    """A farthest-first policy beats nearest-first on a trace built for it,
    so the MIN pin can tell the two apart."""
    reqs = [{0, 1}, {2}, {1}, {0}]
    assert belady_min_loads(reqs, 2) == 4
    assert optimal_loads(reqs, 3, 2) == 4
