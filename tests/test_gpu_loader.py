"""GPU parity of the load-task scheduler (Appendix A, load task scheduler and
preemption): the native scheduler's chunk log must equal the oracle model's
exactly, and every destination unit must hold its agent's bytes."""
import json
import os
import threading
import time

import numpy as np
import pytest

import workloads as W
from gpu_harness import fill_host, log
from oracle.loader import LoaderModel
from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer, PoolMemory

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden", "loader")


class Module:
    """A module's device planes, pinned host copies (filled with the content
    generator) and a destination-unit list per agent (disjoint units)."""

    def __init__(self, units, chunk_bytes, chunk_units, ring, seed):
        units = np.asarray(units, dtype=np.uint32)
        cap = int(units.sum()) + 7
        self.spec = W.PoolSpec(f"m{seed}", cap, list(chunk_bytes), units)
        ub = self.spec.unit_bytes
        self.mem = PoolMemory(self.spec, ring * chunk_units * ub, ring)
        self.content = W.Content(self.spec, seed=seed, pool_index=0)
        fill_host(self.mem, self.content, self.spec)
        rng = np.random.default_rng(seed)
        perm = rng.permutation(cap)[:int(units.sum())].astype(np.int32)
        self.off = np.concatenate([[0], np.cumsum(units)]).astype(np.int64)
        self.lists = perm
        self.dlists = DeviceBuffer(perm.nbytes)
        self.dlists.upload(perm)
        # poison the planes so that every checked byte must have been written
        for p in self.mem.planes:
            p.upload(np.full(p.nbytes, 0xA5, np.uint8))

    def units_ptr(self, a):
        return self.dlists.ptr + 4 * int(self.off[a])

    def check(self, agents, label):
        for a in agents:
            n = int(self.spec.agent_units[a])
            dst = self.lists[self.off[a]:self.off[a] + n]
            got = self.mem.units_bytes(dst)
            exp = self.content.units_bytes(np.full(n, a), np.arange(n))
            assert np.array_equal(got, exp), (label, "bytes of agent", a)

    def free(self):
        self.dlists.free()
        self.mem.free()


def run_both(mods, script, preempt=True, label=""):
    loader = B.Loader([m.mem.desc_args() for m in mods], preempt=preempt)
    model = LoaderModel([m.spec.agent_units for m in mods],
                        [m.mem.staging.nbytes // m.mem.ring_slots // m.spec.unit_bytes
                         for m in mods], preempt=preempt)
    got, exp, done = [], [], set()
    try:
        for op in script:
            if op[0] == "submit":
                _, mod, a, d = op
                loader.submit([(mod, a, d, mods[mod].units_ptr(a))])
                model.submit(mod, a, d)
            else:
                got += loader.pump(op[1])
                exp += model.pump(op[1])
        got += loader.pump(1 << 20)
        exp += model.pump(1 << 20)
        loader.sync()
        assert loader.pending() == (0, 0)
        st = loader.stats()
    finally:
        loader.close()
    assert [tuple(x) for x in got] == [tuple(x) for x in exp], label
    for (m, a, _, _, f) in got:
        if f & B.SS_LOAD_DONE:
            done.add((m, a))
    for i, m in enumerate(mods):
        m.check(sorted(a for (mm, a) in done if mm == i), label)
    return got, st


def test_paper_preemption_sequence():
    fx = json.load(open(os.path.join(GOLD, "preemption.json")))
    mod = Module(fx["agent_units"][0], [4096, 2048], fx["chunk_units"][0], 2, seed=1)
    try:
        log(f"[loader] paper sequence")
        got, st = run_both([mod], [tuple(x) for x in fx["script"]], label="paper")
        assert [list(x) for x in got] == fx["expect"]
        assert st["preemptions"] == 1 and st["completed"] == 2
    finally:
        mod.free()


@pytest.mark.parametrize("preempt", [True, False])
@pytest.mark.parametrize("seed", range(4))
def test_random_scripts(seed, preempt):
    rng = np.random.default_rng(seed)
    n_mod = 1 + seed % 2
    mods = []
    try:
        for k in range(n_mod):
            units = rng.integers(1, 30, size=40)
            mods.append(Module(units, [[4096, 2048], [8192], [1024, 1024, 2048]][k + seed % 2],
                               int(rng.integers(1, 6)), int(rng.integers(1, 4)), seed=10 * seed + k))
        script = []
        for _ in range(120):
            if rng.random() < 0.55:
                m = int(rng.integers(n_mod))
                script.append(("submit", m, int(rng.integers(40)), int(rng.integers(0, 8))))
            else:
                script.append(("pump", int(rng.integers(1, 6))))
        log(f"[loader] random seed={seed} modules={n_mod} preempt={preempt}")
        got, st = run_both(mods, script, preempt=preempt, label=f"seed {seed}")
        if not preempt:
            assert st["preemptions"] == 0
    finally:
        for m in mods:
            m.free()


def test_urgent_task_from_another_thread():
    """A long task is being pumped on a worker thread; an urgent task
    submitted meanwhile runs at the next chunk decision."""
    units = np.array([1200, 6], dtype=np.uint32)
    mod = Module(units, [32768] * 4, 2, 2, seed=7)
    loader = B.Loader([mod.mem.desc_args()])
    out = {}
    try:
        loader.submit([(0, 0, 5, mod.units_ptr(0))])
        th = threading.Thread(target=lambda: out.setdefault("log", loader.pump(1 << 20)))
        th.start()
        t0 = time.time()
        while loader.stats()["chunks"] < 10 and time.time() - t0 < 30:
            time.sleep(0.001)
        loader.submit([(0, 1, 0, mod.units_ptr(1))])
        bound = loader.stats()["chunks"]
        th.join(timeout=60)
        assert not th.is_alive()
        got = out["log"] + loader.pump(1 << 20)     # in case the worker finished first
        loader.sync()
        st = loader.stats()
    finally:
        loader.close()
    first_urgent = next(i for i, e in enumerate(got) if e[1] == 1)
    log(f"[loader] urgent task started at chunk {first_urgent} (bound {bound}) of {len(got)}")
    assert first_urgent <= bound
    if first_urgent < len(got) - 3:         # it arrived while agent 0 was still loading
        assert got[first_urgent][4] & B.SS_LOAD_PREEMPT and st["preemptions"] == 1
    assert st["completed"] == 2
    mod.check([0, 1], "thread")
    mod.free()
