"""The allocation-free entry point ss_interaction_distances_static (static
device scratch instead of a workspace) against ss_interaction_distances with
a workspace, bit for bit, through the C ABI: two calls in a row, the second
with fewer agents, so the second reuses scratch the first left behind."""
import numpy as np
import pytest

from paper_2601_21473_amd import binding as B
from paper_2601_21473_amd.memory import DeviceBuffer

pytestmark = pytest.mark.gpu

MAX_AGENTS = 1 << 20


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert B.device_count() > 0, "GPU tests need a GPU"


def _case(n, seed, tiles):
    rng = np.random.default_rng(seed)
    pos = np.ascontiguousarray(rng.integers(0, tiles, size=(n, 2)).astype(np.int32))
    d_act = rng.integers(0, 1000, size=n).astype(np.uint32)
    return pos, d_act


def _run_both(pos, d_act, velocity, radius, stream):
    n = len(d_act)
    bufs = [DeviceBuffer(8 * n), DeviceBuffer(4 * n), DeviceBuffer(4 * n), DeviceBuffer(4 * n)]
    wsb = B.interaction_distances_workspace(n)
    ws = DeviceBuffer(max(wsb, 4))
    try:
        bufs[0].upload(pos.reshape(-1))
        bufs[1].upload(d_act)
        B.interaction_distances(bufs[0].ptr, bufs[1].ptr, n, velocity, radius, bufs[2].ptr, ws.ptr,
                                wsb, stream)
        B.interaction_distances_static(bufs[0].ptr, bufs[1].ptr, n, velocity, radius, bufs[3].ptr,
                                       stream)
        B.stream_sync(stream)
        ref = bufs[2].download(0, 4 * n).view(np.uint32)
        got = bufs[3].download(0, 4 * n).view(np.uint32)
        return ref, got
    finally:
        for b in bufs + [ws]:
            b.free()


def test_static_matches_workspace_two_calls():
    s = B.Stream()
    try:
        # first call: 50,000 agents (the diffusion workload's count); second:
        # 1,000 agents on a small grid, many of them co-located
        for n, seed, tiles, vel, rad in [(50_000, 3, 2048, 3, 2), (1_000, 4, 40, 1, 0)]:
            pos, d_act = _case(n, seed, tiles)
            ref, got = _run_both(pos, d_act, vel, rad, s.handle)
            assert np.array_equal(got, ref), (n, np.flatnonzero(got != ref)[:5])
            assert (got <= d_act).all()
    finally:
        s.sync()
        s.close()


def test_static_rejects_more_agents_than_its_scratch():
    # checked before any argument is touched or any work is queued
    L = B.load()
    st = L.ss_interaction_distances_static(None, None, MAX_AGENTS + 1, 1, 0, None, None)
    assert st == B.SS_ERR_ARG
    assert "static scratch" in L.ss_last_error().decode()


def test_static_empty_and_bad_arguments():
    L = B.load()
    assert L.ss_interaction_distances_static(None, None, 0, 1, 0, None, None) == B.SS_OK
    assert L.ss_interaction_distances_static(None, None, 10, 0, 0, None, None) == B.SS_ERR_ARG
    assert L.ss_interaction_distances_static(None, None, 10, 1, 0, None, None) == B.SS_ERR_ARG
