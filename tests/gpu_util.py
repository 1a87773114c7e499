"""Helpers for the GPU tests: device buffers and one full restore pass through
the C ABI.  Device memory and streams come from torch; every operation is a
call into libflashrestore."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2509_03047_amd import flashrestore as F


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def to_host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def sums_host(t: torch.Tensor, n: int) -> np.ndarray:
    """(n, 2) int64 device sums -> flat uint64 (sum, wsum, ...) host array."""
    return t[:n].cpu().numpy().view(np.uint64).reshape(-1)


class Restore:
    """Buffers and calls of one pack -> unpack -> verify -> checksum pass."""

    def __init__(self, table, chunk_bytes, src_bytes, dst_bytes, canary=0xA5):
        self.plan = F.Plan(table, chunk_bytes, src_bytes, dst_bytes)
        self.src_bytes, self.dst_bytes = src_bytes, dst_bytes
        # pack must write every payload byte, padding and gaps included
        self.payload = self.plan.empty_payload().fill_(0xEE)
        self.sums = self.plan.empty_sums()
        self.dst = torch.full((max(dst_bytes, 1),), canary, dtype=torch.uint8, device="cuda")
        self.bad = self.plan.empty_bitmap()
        self.n_bad = self.plan.empty_counter()
        self.diff = self.plan.empty_bitmap()
        self.n_diff = self.plan.empty_counter()
        self.csum = self.plan.empty_sums()

    @property
    def n_chunks(self):
        return self.plan.n_chunks

    def pack(self, src):
        self.plan.pack(src, self.payload, self.sums)

    def unpack(self, payload=None, sums=None):
        self.plan.unpack(self.payload if payload is None else payload,
                         self.sums if sums is None else sums, self.dst, self.bad, self.n_bad)

    def verify(self, a, b, sums_a=None, sums_b=None):
        self.plan.verify_replicas(a, b, self.diff, self.n_diff, sums_a, sums_b)

    def checksum(self, base):
        self.plan.checksum_state(base, self.csum)

    def bad_set(self):
        torch.cuda.synchronize()
        return set(int(i) for i in F.bitmap_indices(self.bad, self.n_chunks))

    def diff_set(self):
        torch.cuda.synchronize()
        return set(int(i) for i in F.bitmap_indices(self.diff, self.n_chunks))
