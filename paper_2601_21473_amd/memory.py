"""Device and pinned-host buffers of a pool, allocated through libscalesim.

The library's own allocation calls (thin wrappers over the HIP runtime it is
linked with) keep every buffer and every copy on one HIP runtime instance.
On that runtime both directions of ``hipMemcpyAsync`` run on the copy
engines, leaving the compute units to the pack and unpack kernels.
"""
from __future__ import annotations

import ctypes as C

import numpy as np

from . import binding


class DeviceBuffer:
    def __init__(self, nbytes: int, device: int = 0):
        self.nbytes = int(nbytes)
        self.ptr = binding.device_alloc(self.nbytes, device)

    def upload(self, arr: np.ndarray, offset: int = 0):
        a = np.ascontiguousarray(arr)
        assert offset + a.nbytes <= self.nbytes
        binding.copy(self.ptr + offset, a.ctypes.data, a.nbytes)

    def download(self, offset: int, nbytes: int) -> np.ndarray:
        assert offset + nbytes <= self.nbytes
        out = np.empty(nbytes, dtype=np.uint8)
        binding.copy(out.ctypes.data, self.ptr + offset, nbytes)
        return out

    def free(self):
        if self.ptr:
            binding.device_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class HostBuffer:
    """Pinned host memory with a numpy uint8 view."""

    def __init__(self, nbytes: int):
        self.nbytes = int(nbytes)
        self.ptr = binding.host_alloc(self.nbytes)
        self.np = np.ctypeslib.as_array((C.c_uint8 * self.nbytes).from_address(self.ptr))

    def free(self):
        if self.ptr:
            self.np = None
            binding.host_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class PoolMemory:
    """Buffers of one pool: ``n_planes`` device planes of ``capacity *
    chunk_bytes[c]`` bytes, a device staging buffer and pinned host copies.

    ``host_slots`` bounds the host copies: ``None`` gives every agent its own
    copy; an integer ``k`` gives agents ``k`` distinct copies of the largest
    agent size, agent ``a`` using copy ``a % k`` (many logical agents behind one
    physical copy, as the paper does for adapters); an array gives agent ``a``
    copy ``host_slots[a]`` of the largest agent size."""

    def __init__(self, spec, staging_bytes: int, ring_slots: int, host_slots=None,
                 device: int = 0):
        self.spec = spec
        self.planes = [DeviceBuffer(spec.capacity_units * cb, device) for cb in spec.chunk_bytes]
        self.staging = DeviceBuffer(staging_bytes, device)
        ub = spec.unit_bytes
        units = np.asarray(spec.agent_units, dtype=np.uint64)
        if host_slots is None:
            self.host_off = np.concatenate([[0], np.cumsum(units * ub)[:-1]]).astype(np.uint64)
            host_bytes = int(units.sum()) * ub
        else:
            slot = int(units.max()) * ub
            if np.ndim(host_slots) == 0:
                slot_of = np.arange(len(units), dtype=np.uint64) % np.uint64(host_slots)
            else:
                slot_of = np.asarray(host_slots, dtype=np.uint64)
                assert len(slot_of) == len(units)
            self.host_off = slot_of * np.uint64(slot)
            host_bytes = (int(slot_of.max()) + 1) * slot
        self.host = HostBuffer(host_bytes)
        self.host_np = self.host.np
        self.ring_slots = ring_slots
        self.device = device

    def desc_args(self) -> dict:
        """Keyword arguments of ``binding.make_desc`` for these buffers."""
        s = self.spec
        return dict(capacity_units=s.capacity_units, chunk_bytes=s.chunk_bytes,
                    agent_units=s.agent_units, plane_base=[p.ptr for p in self.planes],
                    host_backing=self.host.ptr, host_bytes=self.host.nbytes,
                    host_off=self.host_off, dev_staging=self.staging.ptr,
                    staging_bytes=self.staging.nbytes, ring_slots=self.ring_slots,
                    device=self.device)

    def make_pool(self, timing: bool = False, direct_bytes: int = 0,
                  poll_wait: bool = False) -> binding.Pool:
        s = self.spec
        return binding.Pool(capacity_units=s.capacity_units, chunk_bytes=s.chunk_bytes,
                            agent_units=s.agent_units,
                            plane_base=[p.ptr for p in self.planes],
                            host_backing=self.host.ptr, host_bytes=self.host.nbytes,
                            host_off=self.host_off, dev_staging=self.staging.ptr,
                            staging_bytes=self.staging.nbytes, ring_slots=self.ring_slots,
                            device=self.device, timing=timing, direct_bytes=direct_bytes,
                            poll_wait=poll_wait)

    def host_copy(self, agent: int) -> np.ndarray:
        """View of an agent's host copy (unit-major, planes in order)."""
        off = int(self.host_off[agent])
        n = int(self.spec.agent_units[agent]) * self.spec.unit_bytes
        return self.host_np[off:off + n]

    def units_bytes(self, units) -> np.ndarray:
        """uint8 [K, unit_bytes] of the given physical units, read from the device
        (whole planes when they are small, else chunk by chunk)."""
        s = self.spec
        units = np.asarray(units, dtype=np.int64)
        out = np.empty((len(units), s.unit_bytes), dtype=np.uint8)
        off = 0
        for c, cb in enumerate(s.chunk_bytes):
            if s.capacity_units * cb <= (256 << 20):
                plane = self.planes[c].download(0, s.capacity_units * cb).reshape(-1, cb)
                out[:, off:off + cb] = plane[units]
            else:
                for k, u in enumerate(units):
                    out[k, off:off + cb] = self.planes[c].download(int(u) * cb, cb)
            off += cb
        return out

    def free(self):
        for b in self.planes + [self.staging, self.host]:
            b.free()
