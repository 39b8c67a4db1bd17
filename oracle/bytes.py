"""Oracle of the bytes one step moves (eviction write-back and load).

TEST INFRASTRUCTURE: used by the tests, the smoke check and the benchmark's
CPU-baseline leg only.

Evicted memory is written back to the agent's host copy and loaded memory is
restored from it rather than recomputed (Section 3.3, eviction paragraph;
Section 4.1, "Baselines", on host-backed prefix nodes).  Content never
changes while it sits on the GPU, so a write-back returns the same bytes
(R9: every eviction writes back).

Only the victims in ``plan.written`` are written back (all victims unless a
dirty mask marked some clean; a clean victim's host copy is already current).

Byte order, for both directions: agents in plan order, then the agent's
logical units j = 0.., then the unit's planes c = 0..; an agent's host copy
holds its units in that order, so an agent's bytes are one contiguous range
of the staging stream.
"""
from __future__ import annotations

import numpy as np


class BytePool:
    """A pool's bytes on the host: plane c is a ``[U, chunk_bytes[c]]`` uint8
    array; unit u's chunk of plane c is row u."""

    def __init__(self, capacity_units: int, chunk_bytes):
        self.chunk_bytes = [int(c) for c in chunk_bytes]
        self.planes = [np.zeros((capacity_units, c), dtype=np.uint8) for c in self.chunk_bytes]
        self.unit_bytes = sum(self.chunk_bytes)

    def gather(self, units, out=None) -> np.ndarray:
        """Staging bytes of the given physical units, unit then plane order
        (into ``out`` when given, a buffer of at least that many bytes)."""
        n = len(units) * self.unit_bytes
        out = (np.empty(n, dtype=np.uint8) if out is None else out[:n])
        out = out.reshape(len(units), self.unit_bytes)
        off = 0
        for c, plane in enumerate(self.planes):
            out[:, off:off + self.chunk_bytes[c]] = plane[np.asarray(units, dtype=np.int64)]
            off += self.chunk_bytes[c]
        return out.reshape(-1)

    def scatter(self, units, data) -> None:
        """Write staging bytes (unit then plane order) into the given units."""
        data = np.asarray(data, dtype=np.uint8).reshape(len(units), self.unit_bytes)
        off = 0
        for c, plane in enumerate(self.planes):
            plane[np.asarray(units, dtype=np.int64)] = data[:, off:off + self.chunk_bytes[c]]
            off += self.chunk_bytes[c]


def apply_step_bytes(bpool: BytePool, plan, agent_units, host_read, host_write,
                     staging_out=None, staging_in=None):
    """Move one step's bytes.

    ``host_write(agent, bytes)`` receives each written-back victim's bytes;
    ``host_read(agent)`` returns a loaded agent's host copy.  Returns the two
    staging streams (evicted, loaded) for comparison; ``staging_out`` and
    ``staging_in`` are optional preallocated byte buffers for them."""
    staging_out = bpool.gather(plan.written_units, out=staging_out)
    pos = 0
    for v in plan.written:
        k = int(agent_units[v]) * bpool.unit_bytes
        host_write(int(v), staging_out[pos:pos + k])
        pos += k
    parts = [np.asarray(host_read(int(a)), dtype=np.uint8) for a in plan.loads]
    n_in = sum(len(x) for x in parts)
    staging_in = (np.empty(n_in, dtype=np.uint8) if staging_in is None else staging_in[:n_in])
    if parts:
        np.concatenate(parts, out=staging_in)
    bpool.scatter(plan.load_units, staging_in)
    return staging_out, staging_in
