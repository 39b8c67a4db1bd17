"""Load-task scheduler oracle (Appendix A, load task scheduler and preemption)."""
import json
import os

import numpy as np

from oracle.loader import DONE, PREEMPT, START, LoaderModel

GOLD = os.path.join(os.path.dirname(__file__), "golden", "loader")


def run_script(model, script):
    log = []
    for op in script:
        if op[0] == "submit":
            model.submit(*op[1:])
        else:
            log += model.pump(op[1])
    return [list(x) for x in log]


def test_paper_preemption_sequence():
    fx = json.load(open(os.path.join(GOLD, "preemption.json")))
    assert fx["cite"]
    m = LoaderModel(fx["agent_units"], fx["chunk_units"])
    assert run_script(m, fx["script"]) == fx["expect"]
    assert m.pending() == 0


def test_without_preemption_the_running_task_finishes_first():
    fx = json.load(open(os.path.join(GOLD, "preemption.json")))
    m = LoaderModel(fx["agent_units"], fx["chunk_units"], preempt=False)
    log = run_script(m, fx["script"])
    assert [(a, f) for _, a, _, _, f in log] == [(7, START), (7, 0), (7, 0), (7, DONE),
                                                 (3, START), (3, DONE)]


def test_equal_distance_does_not_interrupt_but_orders_the_queue():
    m = LoaderModel([[3] * 10], [1])
    m.submit(0, 5, 2)
    assert m.pump(1) == [(0, 5, 0, 1, START)]
    m.submit(0, 3, 2)                      # same distance, smaller id: no interruption
    m.submit(0, 1, 2)
    log = m.pump(100)
    assert [a for _, a, _, _, _ in log] == [5, 5, 1, 1, 1, 3, 3, 3]


def test_updated_distance_reorders_and_interrupts():
    m = LoaderModel([[4, 4, 4]], [1])
    m.submit(0, 0, 1)
    m.submit(0, 1, 3)
    assert m.pump(1) == [(0, 0, 0, 1, START)]
    m.submit(0, 0, 5)                      # the running task's estimate grows past agent 1's
    log = m.pump(100)
    assert log[0] == (0, 1, 0, 1, START | PREEMPT)
    assert [a for _, a, _, _, _ in log] == [1] * 4 + [0] * 3
    assert log[4] == (0, 0, 1, 1, START)   # resumes where it stopped


def test_chunking_and_modules():
    m = LoaderModel([[5, 2], [3]], [2, 4])
    m.submit(0, 0, 4)
    m.submit(1, 0, 4)                      # same distance and agent: module breaks the tie
    m.submit(0, 1, 9)
    log = m.pump(100)
    assert log == [(0, 0, 0, 2, START), (0, 0, 2, 2, 0), (0, 0, 4, 1, DONE),
                   (1, 0, 0, 3, START | DONE), (0, 1, 0, 2, START | DONE)]


def test_resubmission_after_completion_is_a_new_task():
    m = LoaderModel([[2]], [1])
    m.submit(0, 0, 1)
    assert len(m.pump(10)) == 2
    m.submit(0, 0, 1)
    assert m.pump(10) == [(0, 0, 0, 1, START), (0, 0, 1, 1, DONE)]


def test_invariants_random():
    """Every submitted task completes; its chunks cover each unit once in
    order; a task issues a chunk only while no queued task has a strictly
    smaller distance; starts follow key order among queued tasks."""
    rng = np.random.default_rng(0)
    for trial in range(50):
        M = int(rng.integers(1, 3))
        units = [rng.integers(1, 9, size=12).tolist() for _ in range(M)]
        chunks = rng.integers(1, 4, size=M).tolist()
        m = LoaderModel(units, chunks)
        covered = {}
        for _ in range(30):
            if rng.random() < 0.5:
                mod, a = int(rng.integers(M)), int(rng.integers(12))
                m.submit(mod, a, int(rng.integers(0, 6)))
            else:
                dist_before = {k: v[0] for k, v in m.tasks.items()}
                running = m.running
                for (mod, a, first, n, flags) in m.pump(int(rng.integers(1, 5))):
                    covered.setdefault((mod, a), []).append((first, n, flags))
                    if flags & START and running is not None and (mod, a) != running \
                            and running in m.tasks:
                        assert flags & PREEMPT or dist_before.get(running) is None
                    running = None if flags & DONE else (mod, a)
        m.pump(10_000)
        assert m.pending() == 0 and m.running is None
        for (mod, a), ch in covered.items():
            # each run of the task covers consecutive units from 0 to s-1
            firsts = [f for f, _, _ in ch]
            nxt = 0
            for f, n, flags in ch:
                if f == 0 and flags & START:
                    nxt = 0
                assert f == nxt
                nxt = f + n
                if flags & DONE:
                    assert nxt == units[mod][a]
            assert firsts
