"""Oracle of the load-task scheduler with preemption.

TEST INFRASTRUCTURE: imported by the tests and the smoke check only.

Appendix A, "Load task scheduler" and "Preemption support": one centralized
scheduler orders every CPU-to-GPU load by invocation distance; a load runs
as a sequence of transfers and checks a preemption signal between them; a
task that is more urgent than the running one interrupts it, the interrupted
task goes back into the queue (ordered by its possibly updated distance) and
the urgent one runs first.

Readings (reproduced by the HIP library):

* R19 a task loads one agent's memory of one module; it runs as chunks of
  ``chunk_units[module]`` consecutive logical units (the last may be
  shorter); the signal is checked before every chunk.
* R20 queue order is the key (distance, agent, module), smallest first (R4's
  tie rule); the signal fires only when a queued task's distance is strictly
  smaller than the running task's (a task of equal distance is not more
  urgent, so equal distances never interrupt each other).
* R21 an interrupted task keeps its progress and resumes at its next chunk;
  resubmitting a queued or running task only updates its distance; a task
  submitted after its agent's previous task completed is a new task.
* R22 without preemption (a scheduler flag) tasks still start in key order
  but always run to completion.
"""
from __future__ import annotations

START, PREEMPT, DONE = 1, 2, 4


class LoaderModel:
    def __init__(self, agent_units, chunk_units, preempt=True):
        """``agent_units[m][a]`` units of agent a in module m; ``chunk_units[m]``."""
        self.s = [list(map(int, u)) for u in agent_units]
        self.k = list(map(int, chunk_units))
        self.preempt = preempt
        self.tasks = {}          # (module, agent) -> [distance, cursor]
        self.running = None      # (module, agent) or None

    def submit(self, module, agent, distance):
        key = (int(module), int(agent))
        if key in self.tasks:
            self.tasks[key][0] = int(distance)
        else:
            self.tasks[key] = [int(distance), 0]

    def _queued_min(self):
        q = [(d, a, m) for (m, a), (d, _) in self.tasks.items() if (m, a) != self.running]
        return min(q) if q else None

    def pump(self, max_chunks):
        """Chunks issued, each as (module, agent, first unit, units, flags)."""
        log = []
        while len(log) < max_chunks:
            flags = 0
            if self.running is None:
                top = self._queued_min()
                if top is None:
                    break
                self.running = (top[2], top[1])
                flags |= START
            elif self.preempt:
                top = self._queued_min()
                if top is not None and top[0] < self.tasks[self.running][0]:
                    self.running = (top[2], top[1])
                    flags |= START | PREEMPT
            m, a = self.running
            cursor = self.tasks[self.running][1]
            n = min(self.k[m], self.s[m][a] - cursor)
            self.tasks[self.running][1] = cursor + n
            if cursor + n == self.s[m][a]:
                flags |= DONE
                del self.tasks[self.running]
                self.running = None
            log.append((m, a, cursor, n, flags))
        return log

    def pending(self):
        return len(self.tasks)
