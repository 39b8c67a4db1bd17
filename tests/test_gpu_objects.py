"""GPU parity of shared-object distances (Appendix A, fine-grained distance
assignment) against the oracle, bit-exact, through the C ABI."""
import json
import os

import numpy as np
import pytest

import workloads as W
from gpu_harness import log, run_parity
from oracle.objects import object_distances
from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer

pytestmark = pytest.mark.gpu
S = W.SENTINEL


class GpuObjects:
    """Device copies of an object -> agents map and the kernel's outputs."""

    def __init__(self, off, agents, n_agents):
        self.M = len(off) - 1
        self.R = int(off[-1])
        self.N = n_agents
        off = np.ascontiguousarray(off, dtype=np.uint32)
        agents = np.ascontiguousarray(agents, dtype=np.uint32)
        self.bufs = []
        self.off = self._buf(off)
        self.agents = self._buf(agents) if self.R else None
        self.dist = DeviceBuffer(max(4, 4 * n_agents))
        self.act = DeviceBuffer(max(1, n_agents))
        self.od = DeviceBuffer(max(4, 4 * self.M))
        self.oa = DeviceBuffer(max(1, self.M))
        self.wsb = B.object_distances_workspace(self.M, self.R, n_agents)
        self.ws = DeviceBuffer(max(16, self.wsb))
        self.bufs += [self.dist, self.act, self.od, self.oa, self.ws]

    def _buf(self, arr):
        b = DeviceBuffer(max(arr.nbytes, 4))
        if arr.nbytes:
            b.upload(arr)
        self.bufs.append(b)
        return b

    def launch(self, d_ptr, a_ptr, stream=0):
        B.object_distances(self.off.ptr, self.agents.ptr if self.agents else 0, self.M, self.R,
                           d_ptr, a_ptr, self.N, self.od.ptr, self.oa.ptr, self.ws.ptr, self.wsb,
                           stream)

    def run(self, D, act, poison=True):
        if self.N:
            self.dist.upload(np.ascontiguousarray(D, dtype=np.uint32))
            self.act.upload(np.ascontiguousarray(act, dtype=np.uint8))
        if poison:           # every output must be written by the kernels
            self.od.upload(np.full(self.M, 0x5A5A5A5A, np.uint32))
            self.oa.upload(np.full(self.M, 0xA5, np.uint8))
            self.ws.upload(np.full(self.ws.nbytes, 0x77, np.uint8))
        self.launch(self.dist.ptr, self.act.ptr)
        d = self.od.download(0, 4 * self.M).view(np.uint32)
        a = self.oa.download(0, self.M)
        return d, a

    def free(self):
        for b in self.bufs:
            b.free()


def check(off, agents, N, D, act, label, sample=None, seed=0):
    g = GpuObjects(off, agents, N)
    try:
        log(f"[objects] {label}: M={g.M} R={g.R} N={N}")
        d, a = g.run(D, act)
    finally:
        g.free()
    M = len(off) - 1
    if sample is not None and M > sample:       # oracle on a seeded sample of objects
        rng = np.random.default_rng(seed)
        idx = np.unique(np.concatenate([[0, M - 1], rng.choice(M, sample, replace=False)]))
        sub_off = np.concatenate([[0], np.cumsum(off[idx + 1] - off[idx])]).astype(np.int64)
        sub_agents = np.concatenate([agents[off[i]:off[i + 1]] for i in idx])
        ed, ea = object_distances(sub_off, sub_agents, D, act)
        assert np.array_equal(d[idx], ed), label
        assert np.array_equal(a[idx], ea), label
    else:
        ed, ea = object_distances(off, agents, D, act)
        bad = np.flatnonzero((d != ed) | (a != ea))
        assert len(bad) == 0, (label, bad[:8], d[bad[:8]], ed[bad[:8]])
    return d, a


def rand_da(N, rng, p_act=0.05, p_far=0.1, hi=200):
    D = rng.integers(0, hi, size=N).astype(np.uint32)
    D[rng.random(N) < p_far] = S
    act = (rng.random(N) < p_act).astype(np.uint8)
    return D, act


def test_paper_example():
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "objects",
                                     "shared_object_min.json")))
    d, a = check(np.array(fx["obj_off"]), np.array(fx["obj_agents"]), 2,
                 np.array(fx["dist"], np.uint32), np.array(fx["active"], np.uint8), "paper")
    assert d.tolist() == fx["expect_dist"] and a.tolist() == fx["expect_active"]


@pytest.mark.parametrize("n,branch,depth", [(1, 2, 1), (200, 3, 4), (5000, 4, 5), (16384, 4, 6)])
def test_prefix_trees(n, branch, depth):
    rng = np.random.default_rng(n)
    off, agents, _ = W.prefix_tree_objects(n, branch, depth, seed=n)
    for k in range(3):
        D, act = rand_da(n, rng, p_act=[0.0, 0.05, 0.5][k])
        check(off, agents, n, D, act, f"tree n={n} b={branch} depth={depth} k={k}")


def test_skewed_rows_span_many_workgroups():
    rng = np.random.default_rng(7)
    N = 3000
    # one object referenced 100k times, runs of empty objects, then many short ones
    lens = np.concatenate([[100_000], np.zeros(10_000, np.int64), rng.integers(0, 5, 20_000),
                           [0], [5000], np.zeros(3, np.int64)])
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    agents = rng.integers(0, N, size=int(off[-1])).astype(np.uint32)
    for p_act in (0.0, 1e-4, 0.2):
        D, act = rand_da(N, rng, p_act=p_act)
        check(off, agents, N, D, act, f"skewed p_act={p_act}")


def test_edge_cases():
    rng = np.random.default_rng(3)
    # no references at all
    check(np.zeros(5000, np.int64), np.zeros(0, np.uint32), 4, np.arange(4, dtype=np.uint32),
          np.zeros(4, np.uint8), "no refs")
    # one object, ragged sizes around the 2048-item tile
    for R in (1, 2046, 2047, 2048, 2049, 4095, 4097):
        D, act = rand_da(50, rng)
        check(np.array([0, R]), rng.integers(0, 50, R).astype(np.uint32), 50, D, act, f"one R={R}")
    # ids outside [0, N) are ignored
    off = np.array([0, 3, 3, 6])
    agents = np.array([0, 9, 1, 7, 8, 9], np.uint32)
    d, a = check(off, agents, 2, np.array([4, 2], np.uint32), np.array([0, 0], np.uint8),
                 "foreign ids")
    assert d.tolist() == [2, S, S]
    # distances at the extremes and inactive agents at distance 0
    D = np.array([0, S, S - 1, 1], np.uint32)
    check(np.array([0, 1, 2, 4, 6]), np.array([0, 1, 1, 2, 3, 1], np.uint32), 4, D,
          np.zeros(4, np.uint8), "extremes")


def test_large_prefix_tree_sampled():
    n = 262_144
    rng = np.random.default_rng(11)
    off, agents, _ = W.prefix_tree_objects(n, 8, 5, seed=5)
    D, act = rand_da(n, rng, p_act=0.01, hi=1 << 20)
    check(off, agents, n, D, act, f"tree n={n}", sample=3000, seed=1)


def test_object_pool_plans_from_object_distances():
    """A pool of shared objects planned with object distances: the HIP side
    computes them on the device from the agents' trace, the oracle side with
    the oracle; plans, block table and moved bytes must agree."""
    n, T = 300, 40
    off, agents, sizes = W.prefix_tree_objects(n, 3, 3, seed=2)
    M = len(off) - 1
    rng = np.random.default_rng(5)
    act_t = np.zeros((T, n), np.uint8)
    for t in range(T):
        act_t[t, rng.choice(n, 6, replace=False)] = 1
    D_t = W.noisy_distances(W.exact_distances(act_t), 2.0, rng)
    od = np.zeros((T, M), np.uint32)
    oa = np.zeros((T, M), np.uint8)
    for t in range(T):
        od[t], oa[t] = object_distances(off, agents, D_t[t], act_t[t])
    need = max(int(sizes[oa[t].astype(bool)].sum()) for t in range(T))
    spec = W.PoolSpec("objects", need + 40, [64, 32], sizes)
    otrace = W.Trace("objects", M, T, [spec], oa, od, od, {})
    g = GpuObjects(off, agents, n)
    dD = DeviceBuffer(D_t.nbytes)
    dA = DeviceBuffer(act_t.nbytes)
    dD.upload(D_t)
    dA.upload(act_t)

    def inputs(t):
        g.launch(dD.ptr + 4 * n * t, dA.ptr + n * t)
        return g.od.ptr, g.oa.ptr

    try:
        run_parity(otrace, theta=30, steps=T, slot_units=4, label="object pool",
                   device_inputs=inputs)
    finally:
        g.free()
        dD.free()
        dA.free()


def test_bench_forest_sampled():
    """The forest the benchmark times (8 trees x 1M agents, branching 8,
    depth 6), on a seeded sample of objects including every tree's root."""
    trees, n1 = 8, 1_000_000
    off, agents, _ = W.prefix_forest(trees, n1, 8, 6, seed=0)
    rng = np.random.default_rng(17)
    n = trees * n1
    D = rng.integers(1, 1 << 20, size=n).astype(np.uint32)
    act = (rng.random(n) < 0.01).astype(np.uint8)
    g = GpuObjects(off, agents, n)
    try:
        log(f"[objects] forest: M={g.M} R={g.R} N={n}")
        d, a = g.run(D, act)
    finally:
        g.free()
    M = len(off) - 1
    per_tree = M // trees
    idx = np.unique(np.concatenate([np.arange(trees) * per_tree, [M - 1],
                                    rng.choice(M, 4000, replace=False)]))
    sub_off = np.concatenate([[0], np.cumsum(off[idx + 1] - off[idx])]).astype(np.int64)
    sub_agents = np.concatenate([agents[off[i]:off[i + 1]] for i in idx])
    ed, ea = object_distances(sub_off, sub_agents, D, act)
    assert np.array_equal(d[idx], ed) and np.array_equal(a[idx], ea)
    # properties at every object: an active object is at 0; every tree's root
    # holds the minimum of its tree
    assert (d[a == 1] == 0).all()
    for k in range(trees):
        Dk = np.where(act[k * n1:(k + 1) * n1] == 1, 0, D[k * n1:(k + 1) * n1])
        assert d[k * per_tree] == Dk.min()
