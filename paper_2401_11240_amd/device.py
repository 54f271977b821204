"""Device residency of a workload: torch owns the memory, liblora computes.

Uploads the 16-bit bit patterns of a seeded workload into device buffers
(every adapter of a projection packed into one A buffer and one B buffer,
each factor 16-byte aligned), registers one adapter table per projection and
holds the step's batch descriptor.  PyTorch is only the allocator and the
stream owner here.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List

import numpy as np

from . import lora as L
from .workloads import Workload


def _torch():
    import torch
    return torch


def to_device_bits(a: np.ndarray, device):
    """uint16 bit patterns -> int16 device tensor with the same bits."""
    torch = _torch()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).to(device)


def from_device_bits(t) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint16)


@dataclass
class DeviceProjection:
    name: str
    h_in: int
    h_out: int
    x: str
    A_buf: object
    B_buf: object
    A_ptrs: List[int]
    B_ptrs: List[int]
    y: object
    table: int = 0

    def release(self):
        if self.table:
            L.lora_release_adapters(self.table)
            self.table = 0


@dataclass
class DeviceWorkload:
    workload: Workload
    device: object
    batch: L.Batch
    xs: Dict[str, object]
    projections: List[DeviceProjection] = field(default_factory=list)

    def projection(self, name: str) -> DeviceProjection:
        for p in self.projections:
            if p.name == name:
                return p
        raise KeyError(name)

    def release(self):
        for p in self.projections:
            p.release()


def pack_factors(mats: List[np.ndarray], device):
    """One device buffer holding every matrix back to back; returns the buffer
    and the address of each matrix (16-byte aligned: sizes are multiples of 8
    elements)."""
    sizes = [int(m.size) for m in mats]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    flat = np.empty(max(1, int(offs[-1])), dtype=np.uint16)
    for m, o in zip(mats, offs[:-1]):
        flat[o:o + m.size] = np.ascontiguousarray(m, dtype=np.uint16).ravel()
    buf = to_device_bits(flat, device)
    base = buf.data_ptr()
    return buf, [base + 2 * int(o) for o in offs[:-1]]


def upload(w: Workload, device="cuda:0", register: bool = True, stream=None) -> DeviceWorkload:
    torch = _torch()
    dev = torch.device(device)
    xs = {k: to_device_bits(v, dev) for k, v in w.xs.items()}
    dw = DeviceWorkload(workload=w, device=dev, batch=L.Batch(w.seg_offset, w.seg_adapter, w.n_rows),
                        xs=xs)
    for p in w.projections:
        A_buf, A_ptrs = pack_factors(p.A, dev)
        B_buf, B_ptrs = pack_factors(p.B, dev)
        dp = DeviceProjection(p.name, p.h_in, p.h_out, p.x, A_buf, B_buf, A_ptrs, B_ptrs,
                              to_device_bits(p.y, dev))
        if register:
            dp.table = L.lora_register_adapters(dev.index or 0, p.h_in, p.h_out, w.dtype, A_ptrs,
                                                B_ptrs, w.ranks, w.scales, stream)
        dw.projections.append(dp)
    return dw
