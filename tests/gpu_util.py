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

    def __init__(self, table, chunk_bytes, src_bytes, dst_bytes, canary=0xA5, seg=None):
        self.plan = F.Plan(table, chunk_bytes, src_bytes, dst_bytes, seg)
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


def stripe_ranges(n: int, k: int):
    """k contiguous chunk ranges of near-equal size covering [0, n)."""
    edges = [n * i // k for i in range(k + 1)]
    return list(zip(edges[:-1], edges[1:]))


def chunk_payload_offset(plan: F.Plan, entry_of_chunk, c: int):
    """Full-payload offset of global chunk c, None for a derived chunk."""
    e = int(entry_of_chunk[c])
    pay_off, first, _ = plan.entry_layout(e)
    if pay_off == 0xFFFFFFFFFFFFFFFF:
        return None
    return pay_off + (c - first) * plan.info["chunk_bytes"]


def striped_payload(plan: F.Plan, table, src: torch.Tensor, ranges):
    """A multi-donor transfer on one GPU: each contiguous chunk range is
    packed on its own (fr_pack_chunks) and placed in a receive buffer at the
    full-payload offset of its first sent chunk, its sums at its chunk ids.
    Returns (receive buffer, sums, [(range, offset, stripe payload, stripe
    sums)]).  Gap bytes of the receive buffer keep a 0xEE canary."""
    n = plan.n_chunks
    counts = [plan.entry_layout(k)[2] for k in range(len(table))]
    entry_of_chunk = np.repeat(np.arange(len(table)), counts)
    recv = plan.empty_payload().fill_(0xEE)
    sums = plan.empty_sums().fill_(0)
    parts = []
    for a, b in ranges:
        ids = np.arange(a, b, dtype=np.uint32)
        pb = plan.delta_layout(ids)
        sp = torch.empty(max(pb, 16), dtype=torch.uint8, device="cuda")
        ss = torch.empty(max(b - a, 1), 2, dtype=torch.int64, device="cuda")
        plan.pack_chunks(src, ids, sp, ss)
        off = next((o for o in (chunk_payload_offset(plan, entry_of_chunk, int(c)) for c in ids)
                    if o is not None), None)
        if off is not None and pb:
            recv[off:off + pb] = sp[:pb]
        if b > a:
            sums[a:b] = ss[: b - a]
        parts.append(((a, b), off, sp[:pb], ss[: b - a]))
    assert sum(counts) == n
    return recv, sums, parts
