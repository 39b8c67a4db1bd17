"""The C ABI without a GPU: the library loads, exports every function the
header declares, the ctypes mirrors match the C struct layouts, and invalid
arguments are rejected before any device work."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2601_21473_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scalesim.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ss_[a-z_]+)\s*\(", text)))


def test_header_functions_exported():
    L = B.load()
    names = declared_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(B.EXPORTS)


def test_struct_layouts_match_header(tmp_path):
    structs = {"ss_pool_desc": B.ss_pool_desc, "ss_plan_params": B.ss_plan_params,
               "ss_plan": B.ss_plan, "ss_stats": B.ss_stats, "ss_load_task": B.ss_load_task,
               "ss_load_log": B.ss_load_log, "ss_loader_stats": B.ss_loader_stats}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "scalesim.h"', "int main(void){"]
    for sname, cls in structs.items():
        lines.append(f'printf("{sname} size %zu\\n", sizeof({sname}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{sname}.{f} %zu\\n", offsetof({sname}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    got = dict(line.rsplit(" ", 1) for line in out.strip().splitlines())
    for sname, cls in structs.items():
        assert int(got[f"{sname} size"]) == C.sizeof(cls), sname
        for f, _ in cls._fields_:
            assert int(got[f"{sname}.{f}"]) == getattr(cls, f).offset, (sname, f)


def test_constants_match_header():
    text = open(HEADER).read()
    for name in ["SS_OK", "SS_ERR_ARG", "SS_ERR_OVERCOMMIT", "SS_ERR_ORDER", "SS_ERR_HIP",
                 "SS_ERR_NOMEM", "SS_ERR_POISONED"]:
        m = re.search(rf"#define {name}\s+\(?(-?\d+)\)?", text)
        assert int(m.group(1)) == getattr(B, name), name
    for name in ["SS_LOADER_NO_PREEMPT", "SS_LOAD_START", "SS_LOAD_PREEMPT", "SS_LOAD_DONE"]:
        m = re.search(rf"#define {name}\s+(\d+)u", text)
        assert int(m.group(1)) == getattr(B, name), name


def _desc(**kw):
    d = B.ss_pool_desc()
    units = np.ones(4, np.uint32)
    chunks = np.array([64, 32], np.uint64)
    bases = (C.c_void_p * 2)(0x1000, 0x2000)
    keep = [units, chunks, bases]
    d.n_agents = 4
    d.capacity_units = 8
    d.n_planes = 2
    d.plane_base = bases
    d.chunk_bytes = chunks.ctypes.data_as(C.POINTER(C.c_uint64))
    d.agent_units = units.ctypes.data_as(C.POINTER(C.c_uint32))
    d.host_backing = 0x10000
    d.host_bytes = 4 * 96
    d.dev_staging = 0x20000
    d.staging_bytes = 2 * 96
    d.ring_slots = 1
    d.device = 0
    for k, v in kw.items():
        setattr(d, k, v)
    return d, keep


@pytest.mark.parametrize("field,value,msg", [
    ("n_agents", 0, "n_agents"),
    ("capacity_units", 0, "capacity_units"),
    ("n_planes", 0, "n_planes"),
    ("host_backing", None, "host_backing"),
    ("dev_staging", None, "dev_staging"),
    ("ring_slots", 0, "ring_slots"),
    ("flags", 4, "flag"),
    ("host_bytes", 4 * 96 - 16, "exceeds host_bytes"),
    ("staging_bytes", 95, "too small"),
])
def test_create_rejects_bad_descriptor(field, value, msg):
    L = B.load()
    d, keep = _desc(**{field: value})
    h = C.c_void_p()
    st = L.ss_pool_create(C.byref(d), C.byref(h))
    assert st == B.SS_ERR_ARG
    assert msg in L.ss_last_error().decode()
    assert not h.value


def test_create_rejects_bad_chunks_and_units():
    L = B.load()
    d, keep = _desc()
    bad = np.array([64, 24], np.uint64)
    d.chunk_bytes = bad.ctypes.data_as(C.POINTER(C.c_uint64))
    h = C.c_void_p()
    assert L.ss_pool_create(C.byref(d), C.byref(h)) == B.SS_ERR_ARG
    assert "multiple of 16" in L.ss_last_error().decode()
    d, keep = _desc()
    z = np.array([1, 0, 1, 1], np.uint32)
    d.agent_units = z.ctypes.data_as(C.POINTER(C.c_uint32))
    assert L.ss_pool_create(C.byref(d), C.byref(h)) == B.SS_ERR_ARG
    assert "agent_units[1]" in L.ss_last_error().decode()


def test_null_arguments():
    L = B.load()
    assert L.ss_pool_create(None, None) == B.SS_ERR_ARG
    out = B.ss_plan()
    prm = B.ss_plan_params(0, B.SS_NO_BUDGET)
    assert L.ss_plan_step(None, None, None, C.byref(prm), C.byref(out), None) == B.SS_ERR_ARG
    assert L.ss_evict_pack(None, None) == B.SS_ERR_ARG
    assert L.ss_prefetch_unpack(None, None) == B.SS_ERR_ARG
    assert L.ss_reset_stats(None) == B.SS_ERR_ARG
    L.ss_pool_destroy(None)


def test_plumbing_argument_checks():
    L = B.load()
    p = C.c_void_p()
    assert L.ss_device_alloc(0, 0, C.byref(p)) == B.SS_ERR_ARG
    assert L.ss_host_alloc(0, C.byref(p)) == B.SS_ERR_ARG
    assert L.ss_copy(None, None, 16) == B.SS_ERR_ARG
    assert L.ss_device_free(None) == B.SS_OK
    assert L.ss_host_free(None) == B.SS_OK
    assert L.ss_sync(None) == B.SS_ERR_ARG
    n = C.c_int32(-1)
    assert L.ss_device_count(C.byref(n)) == B.SS_OK and n.value >= 0


def test_probe_argument_checks():
    L = B.load()
    ms = C.c_float()
    assert L.ss_probe_copy(None, None, 16, 1, C.byref(ms)) == B.SS_ERR_ARG
    assert L.ss_probe_copy(C.c_void_p(16), C.c_void_p(32), 24, 1, C.byref(ms)) == B.SS_ERR_ARG
    assert L.ss_probe_link(C.c_void_p(16), C.c_void_p(32), 16, 3, 1, C.byref(ms)) == B.SS_ERR_ARG


def test_object_distances_argument_checks():
    L = B.load()
    V = C.c_void_p
    # per 2048 merge items (objects + references) a 16-byte carry record, a
    # 4-byte merge-path coordinate per workgroup boundary (padded to 16 bytes)
    # and an 8-byte word per agent
    ws = lambda blocks, n: 16 * blocks + 4 * ((blocks + 1 + 3) // 4 * 4) + 8 * n
    assert L.ss_object_distances_workspace(1, 0, 0) == ws(1, 0)
    assert L.ss_object_distances_workspace(2048, 0, 5) == ws(1, 5)
    assert L.ss_object_distances_workspace(2048, 1, 7) == ws(2, 7)
    assert L.ss_object_distances_workspace(5000, 100000, 3) == ws((105000 + 2047) // 2048, 3)
    args = lambda **kw: [kw.get(k, d) for k, d in (
        ("off", V(256)), ("agents", V(512)), ("M", 4), ("R", 8), ("dist", V(1024)),
        ("act", V(2048)), ("N", 3), ("od", V(4096)), ("oa", V(8192)), ("ws", V(16384)),
        ("wsb", 1 << 20), ("st", None))]
    assert L.ss_object_distances(*args(M=0)) == B.SS_OK            # nothing to do
    assert L.ss_object_distances(*args(M=1 << 31)) == B.SS_ERR_ARG
    assert L.ss_object_distances(*args(R=1 << 31)) == B.SS_ERR_ARG
    assert L.ss_object_distances(*args(off=None)) == B.SS_ERR_ARG
    assert L.ss_object_distances(*args(agents=None)) == B.SS_ERR_ARG
    assert L.ss_object_distances(*args(ws=None)) == B.SS_ERR_ARG
    assert L.ss_object_distances(*args(wsb=15)) == B.SS_ERR_ARG
    assert "workspace_bytes" in L.ss_last_error().decode()
    # host addresses are never taken for device memory
    assert L.ss_object_distances(*args()) == B.SS_ERR_ARG


def test_estimator_argument_checks():
    L = B.load()
    V = C.c_void_p
    assert L.ss_hop_distances_workspace(1) == 64 + 2 * 256
    assert L.ss_hop_distances_workspace(1000) == 64 + 2 * 8192
    assert L.ss_interaction_distances_workspace(7) == 28
    hop = lambda **kw: [kw.get(k, d) for k, d in (
        ("off", V(256)), ("col", V(512)), ("V", 4), ("E", 8), ("src", V(1024)), ("ns", 1),
        ("mh", 0xFFFFFFFF), ("hops", V(2048)), ("ws", V(4096)), ("wsb", 1 << 20), ("st", None))]
    assert L.ss_hop_distances(*hop(V=0)) == B.SS_OK
    assert L.ss_hop_distances(*hop(V=1 << 31)) == B.SS_ERR_ARG
    assert L.ss_hop_distances(*hop(off=None)) == B.SS_ERR_ARG
    assert L.ss_hop_distances(*hop(src=None)) == B.SS_ERR_ARG
    assert L.ss_hop_distances(*hop(wsb=64)) == B.SS_ERR_ARG
    assert L.ss_hop_distances(*hop()) == B.SS_ERR_ARG          # host addresses
    it = lambda **kw: [kw.get(k, d) for k, d in (
        ("pos", V(256)), ("da", V(512)), ("n", 4), ("v", 1), ("r", 0), ("out", V(1024)),
        ("ws", V(2048)), ("wsb", 16), ("st", None))]
    assert L.ss_interaction_distances(*it(n=0)) == B.SS_OK
    assert L.ss_interaction_distances(*it(v=0)) == B.SS_ERR_ARG
    assert L.ss_interaction_distances(*it(pos=None)) == B.SS_ERR_ARG
    assert L.ss_interaction_distances(*it(wsb=15)) == B.SS_ERR_ARG
    assert L.ss_interaction_distances(*it()) == B.SS_ERR_ARG


def test_stream_event_argument_checks():
    L = B.load()
    assert L.ss_stream_create(None) == B.SS_ERR_ARG
    assert L.ss_event_create(None) == B.SS_ERR_ARG
    assert L.ss_event_record(None, None) == B.SS_ERR_ARG
    ms = C.c_float()
    assert L.ss_event_elapsed(None, None, C.byref(ms)) == B.SS_ERR_ARG
    assert L.ss_stream_destroy(None) == B.SS_OK and L.ss_event_destroy(None) == B.SS_OK


def test_loader_argument_checks():
    L = B.load()
    h = C.c_void_p()
    assert L.ss_loader_create(None, 1, 0, C.byref(h)) == B.SS_ERR_ARG
    d, keep = _desc()
    arr = (B.ss_pool_desc * 1)(d)
    assert L.ss_loader_create(arr, 0, 0, C.byref(h)) == B.SS_ERR_ARG
    assert L.ss_loader_create(arr, 1, 1, C.byref(h)) == B.SS_ERR_ARG       # unknown flag
    bad, keep2 = _desc(ring_slots=0)
    arr2 = (B.ss_pool_desc * 1)(bad)
    assert L.ss_loader_create(arr2, 1, 0, C.byref(h)) == B.SS_ERR_ARG
    assert L.ss_loader_submit(None, None, 0) == B.SS_ERR_ARG
    n = C.c_uint32()
    assert L.ss_loader_pump(None, 1, None, 0, C.byref(n)) == B.SS_ERR_ARG
    assert L.ss_loader_pending(None, None, None) == B.SS_ERR_ARG
    assert L.ss_loader_sync(None) == B.SS_ERR_ARG
    L.ss_loader_destroy(None)


def test_no_device_is_an_argument_error_not_a_crash():
    if B.device_count() > 0:
        pytest.skip("a GPU is present")
    L = B.load()
    d, keep = _desc()
    h = C.c_void_p()
    assert L.ss_pool_create(C.byref(d), C.byref(h)) == B.SS_ERR_ARG
    assert "not present" in L.ss_last_error().decode()
