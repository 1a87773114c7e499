"""ctypes wrapper of the plain-C oracle (fr_oracle.c).  TEST INFRASTRUCTURE ONLY.

Arrays are numpy: arenas and payloads are uint8, sums are uint64 with two
words (sum, wsum) per chunk, bitmaps are uint32.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import LIB, build

_lib = None

ENTRY_FIELDS = [
    ("src_offset", "<u8", 0),
    ("dst_offset", "<u8", 8),
    ("numel", "<u8", 16),
    ("dtype", "<u4", 24),
    ("derive_from", "<i4", 28),
]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        l = C.CDLL(LIB)
        P = C.c_void_p
        u32, u64 = C.c_uint32, C.c_uint64
        l.oro_plan.argtypes = [P, u32, u64, u64, P, P, P, P]
        l.oro_frsum.argtypes = [P, u64, P, P]
        l.oro_rne_bf16.argtypes = [u32]
        l.oro_rne_bf16.restype = C.c_uint16
        l.oro_rne_bf16_array.argtypes = [P, P, u64]
        l.oro_compare_sums.argtypes = [P, P, u64, P, P]
        l.oro_pack.argtypes = [P, u32, u64, u64, P, P, P]
        l.oro_unpack.argtypes = [P, u32, u64, u64, P, P, P, P, P]
        l.oro_verify.argtypes = [P, u32, u64, P, P, P, P, P, P]
        l.oro_checksum.argtypes = [P, u32, u64, P, P]
        l.oro_checksum_chunks.argtypes = [P, u32, u64, P, P, u64, P]
        l.oro_delta_layout.argtypes = [P, u32, u64, u64, P, u64, P, P]
        l.oro_pack_chunks.argtypes = [P, u32, u64, u64, P, P, u64, P, P]
        l.oro_unpack_chunks.argtypes = [P, u32, u64, u64, P, P, P, u64, P, P, P]
        for f in ("oro_plan", "oro_pack", "oro_unpack", "oro_verify", "oro_checksum",
                  "oro_checksum_chunks", "oro_selfcheck", "oro_threads", "oro_delta_layout",
                  "oro_pack_chunks", "oro_unpack_chunks"):
            getattr(l, f).restype = C.c_int
        l.oro_set_threads.argtypes = [C.c_int]
        l.oro_set_threads.restype = None
        if l.oro_selfcheck() != 0:
            raise RuntimeError("oracle needs a little-endian host")
        _lib = l
    return _lib


def _table(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t)
    assert t.dtype.itemsize == 32
    for name, fmt, off in ENTRY_FIELDS:
        f = t.dtype.fields[name]
        assert f[1] == off and f[0] == np.dtype(fmt), name
    return t


def _p(a) -> int:
    return a.ctypes.data if a is not None else 0


def threads() -> int:
    return lib().oro_threads()


def set_threads(n: int) -> None:
    """OpenMP threads of the following oracle calls (timing only)."""
    lib().oro_set_threads(int(n))


# Payload segment alignment: 16 packs the sent entries back to back (the
# default reading of the payload layout); any larger power of two is the
# same rule with wider zero gaps.
SEGMENT = 16


def plan(t: np.ndarray, C_: int, seg: int = SEGMENT):
    """Per-entry chunk counts, chunk bases (n+1), payload offsets, payload bytes."""
    t = _table(t)
    n = len(t)
    nch = np.zeros(n + 1, np.uint64)
    base = np.zeros(n + 1, np.uint64)
    pay = np.zeros(n + 1, np.uint64)
    pb = np.zeros(1, np.uint64)
    if lib().oro_plan(_p(t), n, C_, seg, _p(nch), _p(base), _p(pay), _p(pb)) != 0:
        raise ValueError("bad chunk size or segment alignment")
    return nch[:n], base, pay[:n], int(pb[0])


def frsum(b: bytes | np.ndarray):
    a = np.frombuffer(bytes(b), np.uint8) if not isinstance(b, np.ndarray) else np.ascontiguousarray(b, np.uint8)
    s = np.zeros(2, np.uint64)
    lib().oro_frsum(_p(a), a.size, s.ctypes.data, s.ctypes.data + 8)
    return int(s[0]), int(s[1])


def rne_bf16(u: int) -> int:
    return int(lib().oro_rne_bf16(int(u) & 0xFFFFFFFF))


def rne_bf16_array(u32: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(u32, np.uint32)
    out = np.empty(u.size, np.uint16)
    lib().oro_rne_bf16_array(_p(u), _p(out), u.size)
    return out


def n_chunks(t, C_):
    return int(plan(t, C_)[1][-1])


def pack(t, C_, src: np.ndarray, seg: int = SEGMENT):
    t = _table(t)
    _, base, _, pb = plan(t, C_, seg)
    nc = int(base[-1])
    payload = np.empty(pb, np.uint8)
    sums = np.empty(2 * max(nc, 1), np.uint64)
    if lib().oro_pack(_p(t), len(t), C_, seg, _p(src), _p(payload), _p(sums)) != 0:
        raise RuntimeError("oro_pack")
    return payload, sums[: 2 * nc]


def unpack(t, C_, payload: np.ndarray, sums: np.ndarray, dst: np.ndarray, seg: int = SEGMENT):
    """Writes into dst in place; returns (bitmap, n_bad)."""
    t = _table(t)
    nc = n_chunks(t, C_)
    bitmap = np.zeros(max((nc + 31) // 32, 1), np.uint32)
    nbad = np.zeros(1, np.uint64)
    sums = np.ascontiguousarray(sums, np.uint64)
    if lib().oro_unpack(_p(t), len(t), C_, seg, _p(payload), _p(sums), _p(dst), _p(bitmap),
                        _p(nbad)) != 0:
        raise RuntimeError("oro_unpack")
    return bitmap[: (nc + 31) // 32], int(nbad[0])


def verify(t, C_, a: np.ndarray, b: np.ndarray, with_sums=False):
    t = _table(t)
    nc = n_chunks(t, C_)
    bitmap = np.zeros(max((nc + 31) // 32, 1), np.uint32)
    nd = np.zeros(1, np.uint64)
    sa = np.empty(2 * max(nc, 1), np.uint64) if with_sums else None
    sb = np.empty(2 * max(nc, 1), np.uint64) if with_sums else None
    if lib().oro_verify(_p(t), len(t), C_, _p(a), _p(b), _p(bitmap), _p(nd), _p(sa), _p(sb)) != 0:
        raise RuntimeError("oro_verify")
    out = (bitmap[: (nc + 31) // 32], int(nd[0]))
    if with_sums:
        out += (sa[: 2 * nc], sb[: 2 * nc])
    return out


def checksum(t, C_, base: np.ndarray):
    t = _table(t)
    nc = n_chunks(t, C_)
    sums = np.empty(2 * max(nc, 1), np.uint64)
    if lib().oro_checksum(_p(t), len(t), C_, _p(base), _p(sums)) != 0:
        raise RuntimeError("oro_checksum")
    return sums[: 2 * nc]


def checksum_chunks(t, C_, base: np.ndarray, ids: np.ndarray):
    t = _table(t)
    ids = np.ascontiguousarray(ids, np.uint64)
    sums = np.empty(2 * max(ids.size, 1), np.uint64)
    if lib().oro_checksum_chunks(_p(t), len(t), C_, _p(base), _p(ids), ids.size, _p(sums)) != 0:
        raise RuntimeError("oro_checksum_chunks")
    return sums[: 2 * ids.size]


def compare_sums(sums_a: np.ndarray, sums_b: np.ndarray):
    """(bitmap, count) of the chunks whose (sum, wsum) differ; sums as two
    uint64 words per chunk, as the other calls return them."""
    a = np.ascontiguousarray(sums_a, np.uint64)
    b = np.ascontiguousarray(sums_b, np.uint64)
    if a.size != b.size or a.size % 2:
        raise ValueError("sums of equal chunk counts")
    nc = a.size // 2
    bitmap = np.zeros(max((nc + 31) // 32, 1), np.uint32)
    nd = np.zeros(1, np.uint64)
    if lib().oro_compare_sums(_p(a), _p(b), nc, _p(bitmap), _p(nd)) != 0:
        raise RuntimeError("oro_compare_sums")
    return bitmap[: (nc + 31) // 32], int(nd[0])


def bitmap_to_set(bitmap: np.ndarray, n: int) -> list:
    bits = np.unpackbits(np.ascontiguousarray(bitmap, "<u4").view(np.uint8), bitorder="little")
    return [int(i) for i in np.nonzero(bits[:n])[0]]


NO_PAYLOAD = (1 << 64) - 1


def delta_layout(t, C_, ids, seg: int = SEGMENT):
    """Per-list-position payload offsets (NO_PAYLOAD for derived) and payload bytes."""
    t = _table(t)
    ids = np.ascontiguousarray(ids, np.uint32)
    off = np.zeros(max(ids.size, 1), np.uint64)
    pb = np.zeros(1, np.uint64)
    if lib().oro_delta_layout(_p(t), len(t), C_, seg, _p(ids), ids.size, _p(off), _p(pb)) != 0:
        raise ValueError("bad chunk list")
    return off[: ids.size], int(pb[0])


def pack_chunks(t, C_, src, ids, seg: int = SEGMENT):
    t = _table(t)
    ids = np.ascontiguousarray(ids, np.uint32)
    _, pb = delta_layout(t, C_, ids, seg)
    payload = np.empty(max(pb, 1), np.uint8)
    sums = np.empty(2 * max(ids.size, 1), np.uint64)
    if lib().oro_pack_chunks(_p(t), len(t), C_, seg, _p(src), _p(ids), ids.size, _p(payload),
                             _p(sums)) != 0:
        raise RuntimeError("oro_pack_chunks")
    return payload[:pb], sums[: 2 * ids.size]


def unpack_chunks(t, C_, payload, sums, ids, dst, seg: int = SEGMENT):
    """Writes into dst in place; returns (bitmap over list positions, n_bad)."""
    t = _table(t)
    ids = np.ascontiguousarray(ids, np.uint32)
    bitmap = np.zeros(max((ids.size + 31) // 32, 1), np.uint32)
    nbad = np.zeros(1, np.uint64)
    payload = np.ascontiguousarray(payload, np.uint8)
    if payload.size == 0:
        payload = np.zeros(1, np.uint8)
    sums = np.ascontiguousarray(sums, np.uint64)
    if lib().oro_unpack_chunks(_p(t), len(t), C_, seg, _p(payload), _p(sums), _p(ids), ids.size,
                               _p(dst), _p(bitmap), _p(nbad)) != 0:
        raise RuntimeError("oro_unpack_chunks")
    return bitmap[: (ids.size + 31) // 32], int(nbad[0])
