"""Distance estimators (Section 3.2) against closed forms, brute force and
library routines."""
import math

import numpy as np
import pytest
import scipy.sparse as sp
from scipy.sparse.csgraph import dijkstra

import workloads as W
from oracle.estimators import hop_distances, interaction_distances

S = W.SENTINEL


def csr(edges, V):
    edges = sorted(edges)
    off = np.zeros(V + 1, dtype=np.int64)
    for u, _ in edges:
        off[u + 1] += 1
    return np.cumsum(off), np.array([v for _, v in edges], dtype=np.uint32)


def test_directed_path_and_cycle():
    n = 9
    off, col = csr([(i, i + 1) for i in range(n - 1)], n)
    assert hop_distances(off, col, [0]).tolist() == list(range(n))
    assert hop_distances(off, col, [4]).tolist() == [S] * 4 + list(range(5))
    off, col = csr([(i, (i + 1) % n) for i in range(n)], n)
    assert hop_distances(off, col, [3]).tolist() == [(i - 3) % n for i in range(n)]
    # two sources: the nearer one counts
    assert hop_distances(off, col, [0, 5]).tolist() == [min(i % n, (i - 5) % n) for i in range(n)]


def test_horizon_duplicates_and_foreign_sources():
    n = 6
    off, col = csr([(i, i + 1) for i in range(n - 1)], n)
    assert hop_distances(off, col, [0], max_hops=2).tolist() == [0, 1, 2, S, S, S]
    assert hop_distances(off, col, [0], max_hops=0).tolist() == [0, S, S, S, S, S]
    assert hop_distances(off, col, [2, 2, 99]).tolist() == [S, S, 0, 1, 2, 3]
    assert hop_distances(off, col, []).tolist() == [S] * n


def brute_hops(A, sources, V):
    """Reachability by repeated one-step expansion of the source set."""
    reach = np.zeros(V, dtype=bool)
    reach[[s for s in sources if s < V]] = True
    hops = np.where(reach, 0, S).astype(np.int64)
    k = 0
    while True:
        k += 1
        nxt = (A.T.astype(np.int64) @ reach.astype(np.int64)) > 0
        new = nxt & ~reach
        if not new.any():
            return hops
        hops[new] = k
        reach |= nxt


@pytest.mark.parametrize("seed", range(6))
def test_against_brute_force_and_scipy(seed):
    rng = np.random.default_rng(seed)
    V = int(rng.integers(5, 60))
    m = int(rng.integers(0, 4 * V))
    edges = list({(int(u), int(v)) for u, v in rng.integers(0, V, size=(m, 2))})
    off, col = csr(edges, V)
    src = rng.choice(V, size=int(rng.integers(1, 4)), replace=False)
    got = hop_distances(off, col, src)
    A = np.zeros((V, V), dtype=bool)
    for u, v in edges:
        A[u, v] = True
    assert got.astype(np.int64).tolist() == brute_hops(A, src, V).tolist()
    g = sp.csr_matrix((np.ones(len(col)), col, off), shape=(V, V))
    ref = dijkstra(g, directed=True, unweighted=True, indices=src, min_only=True)
    ref = np.where(np.isinf(ref), S, ref).astype(np.int64)
    assert got.astype(np.int64).tolist() == ref.tolist()


def test_diffusion_graph_against_scipy():
    tr = W.make_trace("diffusion", 0)
    out = tr.meta["out_neighbors"]
    V = out.shape[0]
    off = np.arange(0, 8 * V + 1, 8)
    col = out.reshape(-1).astype(np.uint32)
    src = np.flatnonzero(tr.active[0])
    got = hop_distances(off, col, src)
    g = sp.csr_matrix((np.ones(len(col)), col, off), shape=(V, V))
    ref = dijkstra(g, directed=True, unweighted=True, indices=src, min_only=True)
    ref = np.where(np.isinf(ref), S, ref).astype(np.uint32)
    assert np.array_equal(got, ref)
    finite = got[got != S]
    assert len(finite) > 0.99 * V and finite.max() <= 12   # a well-connected graph


def test_interaction_closed_forms():
    # two agents 10 tiles apart, closing speed 2: interaction in 5 steps
    d = interaction_distances([[0, 0], [10, 0]], [100, 3], velocity=2)
    assert d.tolist() == [5, 3]
    # 3-4-5 triangle, radius 1: floor((5 - 1) / 3) = 1
    d = interaction_distances([[0, 0], [3, 4]], [S, S], velocity=3, radius=1)
    assert d.tolist() == [1, 1]
    # inside the radius: 0; a lone agent keeps its action distance
    assert interaction_distances([[5, 5], [6, 5]], [9, 9], 1, radius=2).tolist() == [0, 0]
    assert interaction_distances([[1, 2]], [7], 1).tolist() == [7]
    # co-located agents
    assert interaction_distances([[4, 4], [4, 4], [40, 40]], [9, 9, 9], 1).tolist() == [0, 0, 9]


def test_interaction_against_real_arithmetic():
    rng = np.random.default_rng(3)
    pos = rng.integers(0, 200, size=(40, 2))
    d_act = rng.integers(0, 60, size=40).astype(np.uint32)
    for v, r in [(1, 0), (3, 0), (2, 5), (7, 2)]:
        got = interaction_distances(pos, d_act, v, r)
        for i in range(40):
            dist = min(math.hypot(*(pos[i] - pos[j])) for j in range(40) if j != i)
            exp = min(int(d_act[i]), int(math.floor(max(0.0, dist - r) / v + 1e-12)))
            assert got[i] == exp
