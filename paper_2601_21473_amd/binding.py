"""ctypes binding of libscalesim (include/scalesim.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels and HIP copies.  Importing this module does not load the library;
the first call does, and raises if ``libscalesim.so`` has not been built
(``python -m paper_2601_21473_amd.build``).  There is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

# SCALESIM_LIB names another build of the library to load instead (for
# example the one with host-side sanitizers, build.build(sanitize=True)).
LIB_PATH = os.environ.get("SCALESIM_LIB") or \
    os.path.join(os.path.dirname(os.path.abspath(__file__)), "libscalesim.so")

SS_OK = 0
SS_ERR_ARG = -1
SS_ERR_OVERCOMMIT = -2
SS_ERR_ORDER = -3
SS_ERR_HIP = -4
SS_ERR_NOMEM = -5
SS_ERR_POISONED = -6
SS_NO_BUDGET = (1 << 64) - 1
SS_NO_DISTANCE = 0xFFFFFFFF
SS_FLAG_TIMING = 1
SS_FLAG_POLL_WAIT = 2

EXPORTS = ["ss_pool_create", "ss_pool_destroy", "ss_plan_step", "ss_evict_pack",
           "ss_prefetch_unpack", "ss_block_table", "ss_block_table_host", "ss_block_table_host_all", "ss_resident_host",
           "ss_get_stats", "ss_reset_stats", "ss_probe_copy", "ss_probe_launch", "ss_probe_link",
           "ss_sync",
           "ss_device_count", "ss_device_alloc", "ss_host_alloc", "ss_device_free", "ss_host_free",
           "ss_copy", "ss_last_error", "ss_object_distances_workspace", "ss_object_distances",
           "ss_probe_object_distances", "ss_hop_distances_workspace", "ss_hop_distances",
           "ss_interaction_distances_workspace", "ss_interaction_distances",
           "ss_stream_create", "ss_stream_destroy", "ss_stream_sync", "ss_event_create",
           "ss_event_destroy", "ss_event_record", "ss_event_elapsed", "ss_loader_create",
           "ss_loader_destroy", "ss_loader_submit", "ss_loader_pump", "ss_loader_pending",
           "ss_loader_sync", "ss_loader_get_stats", "ss_debug_fail_copy",
           "ss_interaction_distances_static"]


class ss_load_task(C.Structure):
    _fields_ = [("module", C.c_uint32), ("agent", C.c_uint32), ("distance", C.c_uint32),
                ("pad", C.c_uint32), ("units", C.c_void_p)]


class ss_load_log(C.Structure):
    _fields_ = [("module", C.c_uint32), ("agent", C.c_uint32), ("first", C.c_uint32),
                ("count", C.c_uint32), ("flags", C.c_uint32), ("pad", C.c_uint32)]


class ss_loader_stats(C.Structure):
    _fields_ = [("submitted", C.c_uint64), ("completed", C.c_uint64), ("chunks", C.c_uint64),
                ("bytes", C.c_uint64), ("preemptions", C.c_uint64)]


class ss_pool_desc(C.Structure):
    _fields_ = [("n_agents", C.c_uint32), ("capacity_units", C.c_uint64),
                ("n_planes", C.c_uint32), ("plane_base", C.POINTER(C.c_void_p)),
                ("chunk_bytes", C.POINTER(C.c_uint64)), ("agent_units", C.POINTER(C.c_uint32)),
                ("host_backing", C.c_void_p), ("host_off", C.POINTER(C.c_uint64)),
                ("host_bytes", C.c_uint64), ("dev_staging", C.c_void_p),
                ("staging_bytes", C.c_uint64), ("ring_slots", C.c_uint32),
                ("device", C.c_int32), ("flags", C.c_uint32), ("direct_bytes", C.c_uint64)]


class ss_plan_params(C.Structure):
    _fields_ = [("threshold", C.c_uint32), ("budget_units", C.c_uint64), ("dirty", C.c_void_p)]


class ss_plan(C.Structure):
    _fields_ = [("n_victims", C.c_uint32), ("n_loads", C.c_uint32), ("n_demand", C.c_uint32),
                ("n_demand_victims", C.c_uint32), ("victims", C.POINTER(C.c_uint32)),
                ("loads", C.POINTER(C.c_uint32)), ("units_out", C.c_uint64),
                ("units_in", C.c_uint64), ("bytes_out", C.c_uint64), ("bytes_in", C.c_uint64),
                ("units_written", C.c_uint64), ("victim_written", C.POINTER(C.c_uint8)),
                ("d_victims", C.c_void_p), ("d_loads", C.c_void_p)]


class ss_stats(C.Structure):
    _fields_ = [("steps", C.c_uint64), ("pack_launches", C.c_uint64),
                ("unpack_launches", C.c_uint64), ("pack_bytes", C.c_uint64),
                ("unpack_bytes", C.c_uint64), ("pack_ms", C.c_double), ("unpack_ms", C.c_double),
                ("d2h_bytes", C.c_uint64), ("h2d_bytes", C.c_uint64), ("d2h_ms", C.c_double),
                ("h2d_ms", C.c_double), ("plan_gpu_ms", C.c_double),
                ("plan_phase_us", C.c_double * 7), ("plan_host_us", C.c_double * 3),
                ("direct_out_launches", C.c_uint64), ("direct_in_launches", C.c_uint64),
                ("direct_out_bytes", C.c_uint64), ("direct_in_bytes", C.c_uint64),
                ("direct_out_ms", C.c_double), ("direct_in_ms", C.c_double),
                ("plan_enqueue_us", C.c_double * 4), ("duplex_launches", C.c_uint64),
                ("duplex_bytes", C.c_uint64), ("duplex_ms", C.c_double)]


class ScaleSimError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"scalesim status {status}: {msg}")
        self.status = status


class OvercommitError(ScaleSimError):
    pass


_lib = None


def load():
    """Load libscalesim.so and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2601_21473_amd.build")
    L = C.CDLL(LIB_PATH)
    P = C.c_void_p
    sig = {
        "ss_pool_create": ([C.POINTER(ss_pool_desc), C.POINTER(P)], C.c_int32),
        "ss_pool_destroy": ([P], None),
        "ss_plan_step": ([P, P, P, C.POINTER(ss_plan_params), C.POINTER(ss_plan), P], C.c_int32),
        "ss_evict_pack": ([P, P], C.c_int32),
        "ss_prefetch_unpack": ([P, P], C.c_int32),
        "ss_block_table": ([P, C.POINTER(P), C.POINTER(P)], C.c_int32),
        "ss_block_table_host": ([P, C.c_uint32, C.POINTER(C.c_int32), C.c_uint32,
                                 C.POINTER(C.c_uint32)], C.c_int32),
        "ss_block_table_host_all": ([P, C.POINTER(C.c_int32), C.c_uint64,
                                     C.POINTER(C.c_uint64)], C.c_int32),
        "ss_resident_host": ([P, C.POINTER(C.c_uint8)], C.c_int32),
        "ss_get_stats": ([P, C.POINTER(ss_stats)], C.c_int32),
        "ss_reset_stats": ([P], C.c_int32),
        "ss_probe_copy": ([P, P, C.c_uint64, C.c_int, C.POINTER(C.c_float)], C.c_int32),
        "ss_probe_launch": ([C.c_int, C.POINTER(C.c_float)], C.c_int32),
        "ss_probe_link": ([P, P, C.c_uint64, C.c_int, C.c_int, C.POINTER(C.c_float)], C.c_int32),
        "ss_sync": ([P], C.c_int32),
        "ss_device_count": ([C.POINTER(C.c_int32)], C.c_int32),
        "ss_device_alloc": ([C.c_int32, C.c_uint64, C.POINTER(P)], C.c_int32),
        "ss_host_alloc": ([C.c_uint64, C.POINTER(P)], C.c_int32),
        "ss_device_free": ([P], C.c_int32),
        "ss_host_free": ([P], C.c_int32),
        "ss_copy": ([P, P, C.c_uint64], C.c_int32),
        "ss_last_error": ([], C.c_char_p),
        "ss_object_distances_workspace": ([C.c_uint32, C.c_uint32, C.c_uint32], C.c_uint64),
        "ss_object_distances": ([P, P, C.c_uint32, C.c_uint32, P, P, C.c_uint32, P, P, P,
                                 C.c_uint64, P], C.c_int32),
        "ss_probe_object_distances": ([P, P, C.c_uint32, C.c_uint32, P, P, C.c_uint32, P, P, P,
                                       C.c_uint64, C.c_int, C.POINTER(C.c_float)], C.c_int32),
        "ss_stream_create": ([C.POINTER(P)], C.c_int32),
        "ss_stream_destroy": ([P], C.c_int32),
        "ss_stream_sync": ([P], C.c_int32),
        "ss_event_create": ([C.POINTER(P)], C.c_int32),
        "ss_event_destroy": ([P], C.c_int32),
        "ss_event_record": ([P, P], C.c_int32),
        "ss_event_elapsed": ([P, P, C.POINTER(C.c_float)], C.c_int32),
        "ss_loader_create": ([C.POINTER(ss_pool_desc), C.c_uint32, C.c_uint32, C.POINTER(P)],
                             C.c_int32),
        "ss_loader_destroy": ([P], None),
        "ss_loader_submit": ([P, C.POINTER(ss_load_task), C.c_uint32], C.c_int32),
        "ss_loader_pump": ([P, C.c_uint32, C.POINTER(ss_load_log), C.c_uint32,
                            C.POINTER(C.c_uint32)], C.c_int32),
        "ss_loader_pending": ([P, C.POINTER(C.c_uint32), C.POINTER(C.c_uint32)], C.c_int32),
        "ss_loader_sync": ([P], C.c_int32),
        "ss_loader_get_stats": ([P, C.POINTER(ss_loader_stats)], C.c_int32),
        "ss_hop_distances_workspace": ([C.c_uint32], C.c_uint64),
        "ss_hop_distances": ([P, P, C.c_uint32, C.c_uint32, P, C.c_uint32, C.c_uint32, P, P,
                              C.c_uint64, P], C.c_int32),
        "ss_debug_fail_copy": ([C.c_uint32], None),
        "ss_interaction_distances_static": ([P, P, C.c_uint32, C.c_uint32, C.c_uint32, P, P],
                                            C.c_int32),
        "ss_interaction_distances_workspace": ([C.c_uint32], C.c_uint64),
        "ss_interaction_distances": ([P, P, C.c_uint32, C.c_uint32, C.c_uint32, P, P, C.c_uint64,
                                      P], C.c_int32),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(status: int):
    if status != SS_OK:
        msg = load().ss_last_error().decode()
        if status == SS_ERR_OVERCOMMIT:
            raise OvercommitError(status, msg)
        raise ScaleSimError(status, msg)


def _u64(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def make_desc(*, capacity_units, chunk_bytes, agent_units, plane_base, host_backing, host_bytes,
              dev_staging, staging_bytes, ring_slots, host_off=None, device=0, flags=0,
              direct_bytes=0):
    """An ``ss_pool_desc`` and the arrays it points to (keep them alive)."""
    chunk = _u64(chunk_bytes)
    units = np.ascontiguousarray(agent_units, dtype=np.uint32)
    bases = (C.c_void_p * len(plane_base))(*[int(b) for b in plane_base])
    hoff = None if host_off is None else _u64(host_off)
    d = ss_pool_desc()
    d.n_agents = len(units)
    d.capacity_units = int(capacity_units)
    d.n_planes = len(chunk)
    d.plane_base = bases
    d.chunk_bytes = chunk.ctypes.data_as(C.POINTER(C.c_uint64))
    d.agent_units = units.ctypes.data_as(C.POINTER(C.c_uint32))
    d.host_backing = int(host_backing)
    d.host_off = None if hoff is None else hoff.ctypes.data_as(C.POINTER(C.c_uint64))
    d.host_bytes = int(host_bytes)
    d.dev_staging = int(dev_staging)
    d.staging_bytes = int(staging_bytes)
    d.ring_slots = int(ring_slots)
    d.device = int(device)
    d.flags = int(flags)
    d.direct_bytes = int(direct_bytes)
    return d, (chunk, units, bases, hoff)


class Pool:
    """One memory module's pool (``ss_pool``).  Pointers are plain integers
    (device addresses, pinned host addresses, hipStream_t handles)."""

    def __init__(self, *, capacity_units, chunk_bytes, agent_units, plane_base, host_backing,
                 host_bytes, dev_staging, staging_bytes, ring_slots, host_off=None, device=0,
                 timing=False, direct_bytes=0, poll_wait=False):
        L = load()
        d, self._keep = make_desc(capacity_units=capacity_units, chunk_bytes=chunk_bytes,
                                  agent_units=agent_units, plane_base=plane_base,
                                  host_backing=host_backing, host_bytes=host_bytes,
                                  dev_staging=dev_staging, staging_bytes=staging_bytes,
                                  ring_slots=ring_slots, host_off=host_off, device=device,
                                  flags=(SS_FLAG_TIMING if timing else 0)
                                  | (SS_FLAG_POLL_WAIT if poll_wait else 0),
                                  direct_bytes=direct_bytes)
        self._chunk = self._keep[0]
        self._units = self._keep[1]
        self.n_agents = len(self._units)
        h = C.c_void_p()
        _check(L.ss_pool_create(C.byref(d), C.byref(h)))
        self._h = h
        self.unit_bytes = int(self._chunk.sum())
        # reused argument structs of ss_plan_step
        self._prm, self._out = ss_plan_params(), ss_plan()
        self._prm_ref, self._out_ref = C.byref(self._prm), C.byref(self._out)
        self._plan = L.ss_plan_step
        self._views = {}            # numpy views of the pool-owned host lists, by address

    def close(self):
        if getattr(self, "_h", None):
            load().ss_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def plan_step(self, distances_ptr: int, active_ptr: int, threshold: int, budget=None,
                  stream: int = 0, dirty_ptr: int = 0, lists: bool = True):
        """``ss_plan_step``; returns a dict with numpy copies of the plan and
        the device addresses of its device mirrors (``d_victims``, ``d_loads``).
        ``distances_ptr``, ``active_ptr`` and ``dirty_ptr`` (the [N] write-back
        mask, 0 = none) are addresses of device or host memory.
        ``lists=False`` returns the counts and byte totals only (no copies)."""
        prm, out = self._prm, self._out
        prm.threshold = int(threshold)
        prm.budget_units = SS_NO_BUDGET if budget is None else int(budget)
        prm.dirty = int(dirty_ptr) or None
        _check(self._plan(self._h, int(distances_ptr), int(active_ptr), self._prm_ref,
                          self._out_ref, int(stream) or None))
        if not lists:
            return {"units_out": out.units_out, "units_in": out.units_in,
                    "bytes_out": out.bytes_out, "bytes_in": out.bytes_in,
                    "n_victims": out.n_victims, "n_loads": out.n_loads}
        nv, nl = out.n_victims, out.n_loads
        victims = self._host_list(out.victims, np.uint32)[:nv].copy()
        loads = self._host_list(out.loads, np.uint32)[:nl].copy()
        written = self._host_list(out.victim_written, np.uint8)[:nv].copy()
        return {"victims": victims, "loads": loads, "n_victims": nv, "n_loads": nl,
                "n_demand": out.n_demand,
                "n_demand_victims": out.n_demand_victims, "units_out": out.units_out,
                "units_in": out.units_in, "bytes_out": out.bytes_out, "bytes_in": out.bytes_in,
                "units_written": out.units_written, "victim_written": written,
                "d_victims": out.d_victims or 0, "d_loads": out.d_loads or 0}

    def _host_list(self, ptr, dtype) -> np.ndarray:
        """A numpy view of N entries of one of the plan's host lists.  The
        lists live in pool-owned host memory that keeps its address for the
        pool's life, so the view is made once per address."""
        addr = C.cast(ptr, C.c_void_p).value
        if not addr:
            return np.zeros(0, dtype)
        v = self._views.get((addr, dtype))
        if v is None:
            ctype = C.c_uint32 if dtype == np.uint32 else C.c_uint8
            v = np.ctypeslib.as_array((ctype * self.n_agents).from_address(addr))
            self._views[(addr, dtype)] = v
        return v

    def evict_pack(self, stream: int = 0):
        _check(load().ss_evict_pack(self._h, int(stream) or None))

    def prefetch_unpack(self, stream: int = 0):
        _check(load().ss_prefetch_unpack(self._h, int(stream) or None))

    def block_table(self):
        """(device pointer of int32 units, device pointer of uint64 agent offsets)."""
        u, o = C.c_void_p(), C.c_void_p()
        _check(load().ss_block_table(self._h, C.byref(u), C.byref(o)))
        return u.value, o.value

    def block_table_host(self, agent: int) -> np.ndarray:
        cap = int(self._units[agent])
        buf = np.empty(cap, dtype=np.int32)
        n = C.c_uint32()
        _check(load().ss_block_table_host(self._h, int(agent),
                                          buf.ctypes.data_as(C.POINTER(C.c_int32)), cap,
                                          C.byref(n)))
        return buf[: n.value]

    def block_table_host_all(self) -> np.ndarray:
        """The whole block table, agent after agent (-1 = not resident)."""
        cap = int(self._units.astype(np.uint64).sum())
        buf = np.empty(cap, dtype=np.int32)
        n = C.c_uint64()
        _check(load().ss_block_table_host_all(self._h, buf.ctypes.data_as(C.POINTER(C.c_int32)),
                                              cap, C.byref(n)))
        return buf[: n.value]

    def resident_host(self) -> np.ndarray:
        out = np.empty(self.n_agents, dtype=np.uint8)
        _check(load().ss_resident_host(self._h, out.ctypes.data_as(C.POINTER(C.c_uint8))))
        return out

    def sync(self):
        """Wait for all of the pool's queued work."""
        _check(load().ss_sync(self._h))

    def stats(self) -> dict:
        s = ss_stats()
        _check(load().ss_get_stats(self._h, C.byref(s)))
        out = {k: getattr(s, k) for k, _ in ss_stats._fields_}
        out["plan_phase_us"] = list(out["plan_phase_us"])
        out["plan_host_us"] = list(out["plan_host_us"])
        out["plan_enqueue_us"] = list(out["plan_enqueue_us"])
        return out

    def reset_stats(self):
        _check(load().ss_reset_stats(self._h))


def debug_fail_copy(n: int):
    """Arm (n >= 1) or disarm (0) the failure of the n-th copy command issued
    from now by the pools' and loaders' data movement (``ss_debug_fail_copy``)."""
    load().ss_debug_fail_copy(int(n))


def device_count() -> int:
    n = C.c_int32()
    _check(load().ss_device_count(C.byref(n)))
    return n.value


def device_alloc(nbytes: int, device: int = 0) -> int:
    p = C.c_void_p()
    _check(load().ss_device_alloc(int(device), int(nbytes), C.byref(p)))
    return p.value


def host_alloc(nbytes: int) -> int:
    p = C.c_void_p()
    _check(load().ss_host_alloc(int(nbytes), C.byref(p)))
    return p.value


def device_free(ptr: int):
    _check(load().ss_device_free(ptr))


def host_free(ptr: int):
    _check(load().ss_host_free(ptr))


def copy(dst: int, src: int, nbytes: int):
    _check(load().ss_copy(int(dst), int(src), int(nbytes)))


def null_stream_sync():
    """Wait for the work queued on the null stream."""
    _check(load().ss_stream_sync(None))


def stream_sync(stream: int = 0):
    """Wait for the work queued on a stream (hipStream_t handle, 0 = null)."""
    _check(load().ss_stream_sync(int(stream) or None))


def probe_copy(dst: int, src: int, nbytes: int, iters: int = 10) -> float:
    ms = C.c_float()
    _check(load().ss_probe_copy(int(dst), int(src), int(nbytes), int(iters), C.byref(ms)))
    return ms.value


def probe_launch(iters: int = 50) -> float:
    """Median host round trip (us) of one empty kernel launch and its wait."""
    us = C.c_float()
    _check(load().ss_probe_launch(int(iters), C.byref(us)))
    return us.value


def probe_link(host: int, dev: int, nbytes: int, direction: int, iters: int = 5) -> float:
    ms = C.c_float()
    _check(load().ss_probe_link(int(host), int(dev), int(nbytes), int(direction), int(iters),
                                C.byref(ms)))
    return ms.value


def object_distances_workspace(n_objects: int, n_refs: int, n_agents: int) -> int:
    return int(load().ss_object_distances_workspace(int(n_objects), int(n_refs), int(n_agents)))


def object_distances(obj_off: int, obj_agents: int, n_objects: int, n_refs: int,
                     distances: int, active: int, n_agents: int, obj_distances: int,
                     obj_active: int, workspace: int, workspace_bytes: int, stream: int = 0):
    """Queue ``ss_object_distances`` (all pointers are device addresses)."""
    _check(load().ss_object_distances(int(obj_off), int(obj_agents), int(n_objects), int(n_refs),
                                      int(distances), int(active), int(n_agents),
                                      int(obj_distances), int(obj_active), int(workspace),
                                      int(workspace_bytes), int(stream)))


def probe_object_distances(obj_off: int, obj_agents: int, n_objects: int, n_refs: int,
                           distances: int, active: int, n_agents: int, obj_distances: int,
                           obj_active: int, workspace: int, workspace_bytes: int,
                           iters: int = 20) -> float:
    """Event time (ms) per ``ss_object_distances`` run, back to back."""
    ms = C.c_float()
    _check(load().ss_probe_object_distances(int(obj_off), int(obj_agents), int(n_objects),
                                            int(n_refs), int(distances), int(active),
                                            int(n_agents), int(obj_distances), int(obj_active),
                                            int(workspace), int(workspace_bytes), int(iters),
                                            C.byref(ms)))
    return ms.value


def hop_distances_workspace(n_vertices: int) -> int:
    return int(load().ss_hop_distances_workspace(int(n_vertices)))


def hop_distances(row_off: int, col: int, n_vertices: int, n_edges: int, sources: int,
                  n_sources: int, max_hops: int, hops: int, workspace: int,
                  workspace_bytes: int, stream: int = 0):
    """Queue ``ss_hop_distances`` (device addresses)."""
    _check(load().ss_hop_distances(int(row_off), int(col), int(n_vertices), int(n_edges),
                                   int(sources), int(n_sources), int(max_hops), int(hops),
                                   int(workspace), int(workspace_bytes), int(stream)))


def interaction_distances_workspace(n_agents: int) -> int:
    return int(load().ss_interaction_distances_workspace(int(n_agents)))


def interaction_distances(pos_xy: int, d_action: int, n_agents: int, velocity: int,
                          radius: int, out: int, workspace: int, workspace_bytes: int,
                          stream: int = 0):
    """Queue ``ss_interaction_distances`` (device addresses)."""
    _check(load().ss_interaction_distances(int(pos_xy), int(d_action), int(n_agents),
                                           int(velocity), int(radius), int(out), int(workspace),
                                           int(workspace_bytes), int(stream)))


def interaction_distances_static(pos_xy: int, d_action: int, n_agents: int, velocity: int,
                                 radius: int, out: int, stream: int = 0):
    """Queue ``ss_interaction_distances_static`` (device addresses; no
    workspace: the library's static scratch, at most 1,048,576 agents)."""
    _check(load().ss_interaction_distances_static(int(pos_xy), int(d_action), int(n_agents),
                                                  int(velocity), int(radius), int(out),
                                                  int(stream)))


class Stream:
    """A non-blocking HIP stream at the default priority (``handle`` is the
    hipStream_t to pass as a call's ``stream``)."""

    def __init__(self):
        self.stream = C.c_void_p()
        _check(load().ss_stream_create(C.byref(self.stream)))

    @property
    def handle(self) -> int:
        return self.stream.value or 0

    def sync(self):
        _check(load().ss_stream_sync(self.stream))

    def close(self):
        if self.stream.value:
            load().ss_stream_destroy(self.stream)
            self.stream = C.c_void_p()


class EventTimer:
    """Event time of work queued on one library stream:
    ``with EventTimer() as t: f(t.stream)`` then ``t.ms``."""

    def __init__(self):
        L = load()
        self.stream, self._a, self._b = C.c_void_p(), C.c_void_p(), C.c_void_p()
        _check(L.ss_stream_create(C.byref(self.stream)))
        _check(L.ss_event_create(C.byref(self._a)))
        _check(L.ss_event_create(C.byref(self._b)))
        self.ms = None

    def __enter__(self):
        _check(load().ss_event_record(self._a, self.stream))
        return self

    def __exit__(self, *exc):
        L = load()
        if exc[0] is None:
            _check(L.ss_event_record(self._b, self.stream))
            ms = C.c_float()
            _check(L.ss_event_elapsed(self._a, self._b, C.byref(ms)))
            self.ms = ms.value
        else:
            L.ss_stream_sync(self.stream)
        return False

    @property
    def handle(self) -> int:
        return self.stream.value or 0

    def close(self):
        L = load()
        L.ss_event_destroy(self._a)
        L.ss_event_destroy(self._b)
        L.ss_stream_destroy(self.stream)


SS_LOADER_NO_PREEMPT = 2
SS_LOAD_START, SS_LOAD_PREEMPT, SS_LOAD_DONE = 1, 2, 4


class Loader:
    """The load-task scheduler (``ss_loader``) over one or more modules, each
    given as the keyword arguments of ``make_desc``."""

    def __init__(self, modules, preempt=True):
        L = load()
        descs, self._keep = [], []
        for m in modules:
            d, keep = make_desc(**m)
            descs.append(d)
            self._keep.append(keep)
        arr = (ss_pool_desc * len(descs))(*descs)
        h = C.c_void_p()
        _check(L.ss_loader_create(arr, len(descs), 0 if preempt else SS_LOADER_NO_PREEMPT,
                                  C.byref(h)))
        self._h = h

    def submit(self, tasks):
        """``tasks``: iterable of (module, agent, distance, units device pointer)."""
        tasks = list(tasks)
        arr = (ss_load_task * max(1, len(tasks)))()
        for i, (m, a, d, u) in enumerate(tasks):
            arr[i] = ss_load_task(int(m), int(a), int(d), 0, int(u))
        _check(load().ss_loader_submit(self._h, arr, len(tasks)))

    def pump(self, max_chunks):
        """Issue up to ``max_chunks`` chunks; returns their log as tuples
        (module, agent, first, count, flags)."""
        cap = int(max_chunks)
        log = (ss_load_log * max(1, min(cap, 1 << 20)))()
        n = C.c_uint32()
        _check(load().ss_loader_pump(self._h, cap, log, min(cap, 1 << 20), C.byref(n)))
        return [(e.module, e.agent, e.first, e.count, e.flags) for e in log[:min(n.value, cap)]]

    def pending(self):
        q, r = C.c_uint32(), C.c_uint32()
        _check(load().ss_loader_pending(self._h, C.byref(q), C.byref(r)))
        return q.value, r.value

    def sync(self):
        _check(load().ss_loader_sync(self._h))

    def stats(self) -> dict:
        st = ss_loader_stats()
        _check(load().ss_loader_get_stats(self._h, C.byref(st)))
        return {k: getattr(st, k) for k, _ in st._fields_}

    def close(self):
        if getattr(self, "_h", None):
            load().ss_loader_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
