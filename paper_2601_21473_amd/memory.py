"""Device and pinned-host buffers for a pool, allocated with PyTorch.

PyTorch is used here only as an allocator (HBM tensors, pinned host tensors)
and for stream handles; the library never sees a torch type, only addresses.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding


class PoolMemory:
    """Buffers of one pool: ``n_planes`` device planes of ``capacity *
    chunk_bytes[c]`` bytes, a device staging buffer and pinned host copies.

    ``host_slots`` bounds the host copies: ``None`` gives every agent its own
    copy; an integer ``k`` gives agents ``k`` distinct copies of the largest
    agent size, agent ``a`` using copy ``a % k`` (many logical agents behind one
    physical copy, as the paper does for adapters)."""

    def __init__(self, spec, staging_bytes: int, ring_slots: int, host_slots=None,
                 device: int = 0):
        dev = torch.device("cuda", device)
        self.spec = spec
        self.planes = [torch.empty(spec.capacity_units * cb, dtype=torch.uint8, device=dev)
                       for cb in spec.chunk_bytes]
        self.staging = torch.empty(staging_bytes, dtype=torch.uint8, device=dev)
        ub = spec.unit_bytes
        units = np.asarray(spec.agent_units, dtype=np.uint64)
        if host_slots is None:
            self.host_off = np.concatenate([[0], np.cumsum(units * ub)[:-1]]).astype(np.uint64)
            host_bytes = int(units.sum()) * ub
        else:
            slot = int(units.max()) * ub
            self.host_off = (np.arange(len(units), dtype=np.uint64) % np.uint64(host_slots)) * \
                np.uint64(slot)
            host_bytes = int(host_slots) * slot
        self.host = torch.empty(host_bytes, dtype=torch.uint8, pin_memory=True)
        self.host_np = self.host.numpy()
        self.ring_slots = ring_slots
        self.device = device

    def make_pool(self, timing: bool = False) -> binding.Pool:
        s = self.spec
        return binding.Pool(capacity_units=s.capacity_units, chunk_bytes=s.chunk_bytes,
                            agent_units=s.agent_units,
                            plane_base=[p.data_ptr() for p in self.planes],
                            host_backing=self.host.data_ptr(), host_bytes=self.host.numel(),
                            host_off=self.host_off, dev_staging=self.staging.data_ptr(),
                            staging_bytes=self.staging.numel(), ring_slots=self.ring_slots,
                            device=self.device, timing=timing)

    def host_copy(self, agent: int) -> np.ndarray:
        """View of an agent's host copy (unit-major, planes in order)."""
        off = int(self.host_off[agent])
        n = int(self.spec.agent_units[agent]) * self.spec.unit_bytes
        return self.host_np[off:off + n]

    def unit_chunk(self, unit: int, plane: int) -> torch.Tensor:
        cb = self.spec.chunk_bytes[plane]
        return self.planes[plane][unit * cb:(unit + 1) * cb]
