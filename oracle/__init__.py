"""CPU oracle of the invocation-distance memory manager's per-step hot path.

TEST INFRASTRUCTURE, not product code.  It is a plain, slow, obviously
checkable restatement of the method (plan, block-table update and the bytes
moved) that the HIP library is compared against.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import it.  It shares no code with the HIP path; both read their inputs from
the seeded generators in ``workloads``.

Pins (see ``tests/test_oracle_*.py``): the paper's worked examples, Belady
MIN and an exhaustive optimum on unit-size traces, an independent closed-form
statement of the prefetch rule on variable sizes, and the invariants I1-I7
on every step of every workload.
"""
from .policy import OraclePool, Plan, OvercommitError, run_trace, SENTINEL
from .bytes import BytePool, apply_step_bytes
