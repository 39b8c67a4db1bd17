"""The seeded input generators: shapes, capacity, distance definition."""
import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("name", ["tiny", "roundrobin", "bursty", "zipf_lora"])
def test_shapes_and_determinism(name):
    a = W.make_trace(name, 0)
    b = W.make_trace(name, 0)
    assert np.array_equal(a.active, b.active) and np.array_equal(a.dist, b.dist)
    assert a.active.shape == (a.n_steps, a.n_agents) == a.dist.shape
    for p in a.pools:
        assert p.agent_units.shape == (a.n_agents,) and p.agent_units.min() >= 1


def test_exact_distance_definition_brute_force():
    rng = np.random.default_rng(3)
    act = (rng.random((30, 7)) < 0.2).astype(np.uint8)
    d = W.exact_distances(act)
    for t in range(30):
        for a in range(7):
            later = [u for u in range(t + 1, 30) if act[u, a]]
            assert d[t, a] == (later[0] - t if later else W.SENTINEL)


def test_noisy_distances_keep_sentinel_and_floor():
    rng = np.random.default_rng(0)
    dt = np.array([[1, 5, W.SENTINEL, 100]] * 50, dtype=np.uint32)
    dn = W.noisy_distances(dt, 2.0, rng)
    assert (dn[:, 2] == W.SENTINEL).all() and (dn[:, [0, 1, 3]] >= 1).all()
    assert abs(dn[:, 3].astype(float).mean() - 100) < 2


def test_config_sizes():
    tr = W.make_trace("roundrobin", 0)
    p = tr.pools[0]
    assert p.unit_bytes == 2 * 1024 * 1024 and p.n_planes == 64 and p.capacity_units == 19073
    assert 0.03 < tr.active.mean() < 0.07
    z = W.make_trace("zipf_lora", 0)
    assert z.pools[1].unit_bytes == 83886080 and z.pools[1].n_planes == 448
    assert min(z.pools[1].chunk_bytes) == 32 * 1024 and max(z.pools[1].chunk_bytes) == 448 * 1024


def test_lora_sizes_for_ranks():
    per = {r: sum(W.lora_chunk_bytes(16, 2048, 8192, 512, r)) for r in (8, 16, 64)}
    assert per == {8: 11272192, 16: 22544384, 64: 90177536}


def test_splitmix64_reference_values():
    # first outputs of the SplitMix64 generator seeded with 0 (the state
    # advances by the golden-gamma constant before mixing)
    gamma = 0x9E3779B97F4A7C15
    xs = np.array([0, gamma, (2 * gamma) % (1 << 64)], dtype=np.uint64)
    out = W.splitmix64(xs)
    assert [int(x) for x in out] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_content_distinguishes_chunks():
    tr = W.make_trace("tiny", 0)
    c = W.Content(tr.pools[0])
    a = c.chunk(3, 2, 1)
    assert not np.array_equal(a, c.chunk(3, 2, 0))
    assert not np.array_equal(a, c.chunk(3, 1, 1))
    assert not np.array_equal(a, c.chunk(2, 2, 1))
    full = c.agent_bytes(3)
    ub = tr.pools[0].unit_bytes
    assert np.array_equal(full[2 * ub + 4096: 2 * ub + 8192], a)
