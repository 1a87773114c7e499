"""Python binding of libflashrestore (ctypes; argument marshalling only).

Every function here has the name of the C entry point it calls and does no
computation of its own: all work happens in the gfx950 kernels behind the
C ABI.  PyTorch is used only for device memory (``torch.empty(...,
device="cuda")``) and for the current stream.  There is no fallback: if the
shared library is missing or fails to load, importing this module raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libflashrestore.so")

FR_F32 = 1
FR_BF16 = 2
FR_OK = 0
STATUS = {
    0: "FR_OK",
    -1: "FR_E_INVAL",
    -2: "FR_E_ALIGN",
    -3: "FR_E_RANGE",
    -4: "FR_E_OVERLAP",
    -5: "FR_E_NOMEM",
    -6: "FR_E_DEVICE",
    -7: "FR_E_DEVICE_MISMATCH",
}
NO_PAYLOAD = (1 << 64) - 1

# fr_tensor_desc: 32 bytes.
DESC_DTYPE = np.dtype(
    [("src_offset", "<u8"), ("dst_offset", "<u8"), ("numel", "<u8"), ("dtype", "<u4"), ("derive_from", "<i4")]
)
SUM_BYTES = 16  # fr_chunk_sum


class fr_plan_info(C.Structure):
    _fields_ = [
        ("n_entries", C.c_uint64),
        ("chunk_bytes", C.c_uint64),
        ("n_chunks", C.c_uint64),
        ("payload_bytes", C.c_uint64),
        ("bitmap_words", C.c_uint64),
        ("src_arena_bytes", C.c_uint64),
        ("dst_arena_bytes", C.c_uint64),
        ("state_bytes", C.c_uint64),
        ("device", C.c_int64),
        ("segment_align", C.c_uint64),
        ("delta_payload_max", C.c_uint64),
        ("pack_walk", C.c_uint32),
        ("unpack_walk", C.c_uint32),
        ("tile_pack", C.c_uint32),
        ("tile_unpack", C.c_uint32),
        ("tile_verify", C.c_uint32),
        ("tile_checksum", C.c_uint32),
    ]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class fr_decision(C.Structure):
    _fields_ = [
        ("resume_step", C.c_int64),
        ("action", C.c_int32),
        ("n_failed", C.c_uint32),
        ("n_waiting", C.c_uint32),
        ("reserved", C.c_uint32),
    ]


class fr_layout3d(C.Structure):
    _fields_ = [("tp", C.c_uint32), ("pp", C.c_uint32), ("dp", C.c_uint32), ("shard", C.c_uint32),
                ("zero_stage", C.c_uint32), ("reserved", C.c_uint32)]


ACTIONS = {0: "continue", 1: "wait", 2: "stop_and_restore", 3: "checkpoint_fallback", 4: "inconsistent"}


class FlashRestoreError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        name = STATUS.get(status, str(status))
        msg = _lib.fr_strerror(status).decode()
        if status == -6:
            msg += f" (hipError {_lib.fr_last_hip_error()})"
        super().__init__(f"{where}: {name}: {msg}")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2509_03047_amd.build` "
            "(or __graft_entry__.build()) first"
        )
    lib = C.CDLL(LIB_PATH)
    P, u32, u64, i32 = C.c_void_p, C.c_uint32, C.c_uint64, C.c_int
    sig = {
        "fr_plan_create": [P, u32, u64, u64, u64, C.POINTER(P)],
        "fr_plan_create_ex": [P, u32, u64, u64, u64, u64, C.POINTER(P)],
        "fr_plan_get_info": [P, C.POINTER(fr_plan_info)],
        "fr_plan_chunk_of": [P, u32, u64, C.POINTER(u64)],
        "fr_plan_entry_layout": [P, u32, C.POINTER(u64), C.POINTER(u64), C.POINTER(u64)],
        "fr_plan_destroy": [P],
        "fr_layout_query": [P, u32, u64, u64, u64, u64, C.POINTER(fr_plan_info), P, P],
        "fr_pack_state": [P, P, P, u64, P, P],
        "fr_unpack_state": [P, P, P, P, P, P, P],
        "fr_verify_replicas": [P, P, P, P, P, P, P, P],
        "fr_verify_replicas_noalloc": [P, P, P, P, P, P, P, P],
        "fr_compare_sums": [P, P, P, P, P, P],
        "fr_checksum_state": [P, P, P, P],
        "fr_delta_layout": [P, P, u64, C.POINTER(u64)],
        "fr_pack_chunks": [P, P, P, u64, P, u64, P, P],
        "fr_unpack_chunks": [P, P, u64, P, P, u64, P, P, P, P],
        "fr_pack_flagged": [P, P, P, P, u64, P, P, P],
        "fr_unpack_flagged": [P, P, u64, P, P, P, P, P, P],
        "fr_tracker_create": [u32, P, C.c_double, C.c_double, C.POINTER(P)],
        "fr_tracker_destroy": [P],
        "fr_tracker_heartbeat": [P, u32, C.c_int64, C.c_double],
        "fr_tracker_report_failure": [P, u32, C.c_double],
        "fr_tracker_decide": [P, C.c_double, C.POINTER(fr_decision)],
        "fr_tracker_failed_ranks": [P, C.c_double, P, u32, C.POINTER(u32)],
        "fr_tracker_donors": [P, C.c_double, P],
        "fr_layout_rank_coords": [P, u32, P],
        "fr_layout_donors": [P, P, P],
        "fr_layout_state_table": [P, u32, P, u32, P, u32, C.POINTER(u32), C.POINTER(u64)],
        "fr_strerror": [i32],
        "fr_last_hip_error": [],
        "fr_abi_version": [],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.fr_strerror.restype = C.c_char_p
    if lib.fr_abi_version() != 6:
        raise ImportError("libflashrestore ABI version mismatch")
    return lib


_lib = _load()

EXPORTED = (
    "fr_plan_create", "fr_plan_create_ex", "fr_plan_get_info", "fr_plan_chunk_of", "fr_plan_entry_layout",
    "fr_plan_destroy", "fr_layout_query", "fr_pack_state", "fr_unpack_state",
    "fr_verify_replicas", "fr_verify_replicas_noalloc", "fr_compare_sums", "fr_checksum_state",
    "fr_delta_layout",
    "fr_pack_chunks", "fr_unpack_chunks", "fr_pack_flagged", "fr_unpack_flagged",
    "fr_tracker_create", "fr_tracker_destroy", "fr_tracker_heartbeat",
    "fr_tracker_report_failure", "fr_tracker_decide", "fr_tracker_failed_ranks", "fr_tracker_donors",
    "fr_layout_rank_coords", "fr_layout_donors", "fr_layout_state_table",
    "fr_strerror", "fr_last_hip_error", "fr_abi_version",
)


def _check(rc: int, where: str):
    if rc != FR_OK:
        raise FlashRestoreError(rc, where)


def as_table(table) -> np.ndarray:
    """A contiguous fr_tensor_desc array (any structured array with the same
    field names, or rows of (src_offset, dst_offset, numel, dtype, derive_from))."""
    if isinstance(table, np.ndarray) and table.dtype.names:
        out = np.zeros(len(table), dtype=DESC_DTYPE)
        for f in DESC_DTYPE.names:
            out[f] = table[f]
        return out
    return np.array([tuple(r) for r in table], dtype=DESC_DTYPE)


def _ptr(x) -> int | None:
    """Device address of a torch tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _dev(x, need: int, name: str) -> int | None:
    """Address of a device buffer argument that the call accesses for `need`
    bytes.  The library checks that a buffer lies inside one HIP allocation,
    but torch carves many tensors out of one allocation, so a tensor's own
    extent is checked here: it must be a contiguous CUDA tensor of at least
    `need` bytes (ValueError otherwise).  An int is a raw device address whose
    extent the caller vouches for; None is NULL."""
    if x is None or isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError(f"{name}: not a device tensor")
    if not x.is_contiguous():
        raise ValueError(f"{name}: not contiguous")
    nb = x.numel() * x.element_size()
    if nb < need:
        raise ValueError(f"{name}: {nb} bytes, the call accesses {need}")
    return x.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


# Default payload segment alignment (fr_plan_create): segments back to back
# at 16-byte alignment.
SEGMENT_ALIGN = 16


def fr_layout_query(table, chunk_bytes: int, src_arena_bytes: int, dst_arena_bytes: int,
                    segment_align: int = SEGMENT_ALIGN):
    """Host-only validation and layout: (info dict, payload offsets, chunk bases)."""
    t = as_table(table)
    info = fr_plan_info()
    pay = np.zeros(max(len(t), 1), np.uint64)
    base = np.zeros(len(t) + 1, np.uint64)
    rc = _lib.fr_layout_query(t.ctypes.data if len(t) else None, len(t), chunk_bytes,
                              src_arena_bytes, dst_arena_bytes, segment_align, C.byref(info),
                              pay.ctypes.data, base.ctypes.data)
    _check(rc, "fr_layout_query")
    return info.as_dict(), pay[: len(t)], base


class Plan:
    """A plan bound to the current HIP device: ``fr_plan_create``, or
    ``fr_plan_create_ex`` when a payload segment alignment is given."""

    def __init__(self, table, chunk_bytes: int, src_arena_bytes: int, dst_arena_bytes: int,
                 segment_align: int | None = None):
        self._h = None
        self.table = as_table(table)
        h = C.c_void_p()
        tp = self.table.ctypes.data if len(self.table) else None
        if segment_align is None:
            rc = _lib.fr_plan_create(tp, len(self.table), chunk_bytes, src_arena_bytes, dst_arena_bytes,
                                     C.byref(h))
        else:
            rc = _lib.fr_plan_create_ex(tp, len(self.table), chunk_bytes, src_arena_bytes,
                                        dst_arena_bytes, segment_align, C.byref(h))
        _check(rc, "fr_plan_create")
        self._h = h
        info = fr_plan_info()
        _check(_lib.fr_plan_get_info(self._h, C.byref(info)), "fr_plan_get_info")
        self.info = info.as_dict()

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("plan destroyed")
        return self._h

    def destroy(self):
        if self._h is not None:
            _lib.fr_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    # -- sizes
    @property
    def n_chunks(self) -> int:
        return self.info["n_chunks"]

    @property
    def payload_bytes(self) -> int:
        return self.info["payload_bytes"]

    @property
    def bitmap_words(self) -> int:
        return self.info["bitmap_words"]

    def chunk_of(self, entry: int, byte_in_entry: int) -> int:
        c = C.c_uint64()
        _check(_lib.fr_plan_chunk_of(self.handle, entry, byte_in_entry, C.byref(c)), "fr_plan_chunk_of")
        return c.value

    def entry_layout(self, entry: int):
        p, f, n = C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(_lib.fr_plan_entry_layout(self.handle, entry, C.byref(p), C.byref(f), C.byref(n)),
               "fr_plan_entry_layout")
        return p.value, f.value, n.value

    # -- device buffers (torch allocations, uint8 / int64 / int32)
    def empty_payload(self, device="cuda"):
        import torch

        return torch.empty(max(self.payload_bytes, 1), dtype=torch.uint8, device=device)

    def empty_sums(self, device="cuda"):
        import torch

        return torch.empty(max(self.n_chunks, 1), 2, dtype=torch.int64, device=device)

    def empty_bitmap(self, device="cuda"):
        import torch

        return torch.empty(max(self.bitmap_words, 1), dtype=torch.int32, device=device)

    def empty_counter(self, device="cuda"):
        import torch

        return torch.empty(1, dtype=torch.int64, device=device)

    # -- operations
    def pack(self, src, payload, sums, stream=None, payload_cap=None):
        return fr_pack_state(self, src, payload, payload_cap, sums, stream)

    def unpack(self, payload, sums, dst, bitmap, n_bad, stream=None, sync=False):
        return fr_unpack_state(self, payload, sums, dst, bitmap, n_bad, stream, sync)

    def verify_replicas(self, a, b, bitmap, n_diff, sums_a=None, sums_b=None, stream=None, sync=False):
        return fr_verify_replicas(self, a, b, bitmap, n_diff, sums_a, sums_b, stream, sync)

    def verify_replicas_noalloc(self, a, b, bitmap, n_diff, sums_a=None, sums_b=None, stream=None,
                                sync=False):
        return fr_verify_replicas_noalloc(self, a, b, bitmap, n_diff, sums_a, sums_b, stream, sync)

    def compare_sums(self, sums_a, sums_b, bitmap, n_diff, stream=None, sync=False):
        return fr_compare_sums(self, sums_a, sums_b, bitmap, n_diff, stream, sync)

    def checksum_state(self, base, sums, stream=None):
        return fr_checksum_state(self, base, sums, stream)

    def delta_layout(self, chunk_ids) -> int:
        return fr_delta_layout(self, chunk_ids)

    def pack_chunks(self, src, chunk_ids, payload, sums, stream=None, payload_cap=None):
        return fr_pack_chunks(self, src, chunk_ids, payload, payload_cap, sums, stream)

    def unpack_chunks(self, payload, sums, chunk_ids, dst, bitmap, n_bad, stream=None, payload_bytes=None,
                      sync=False):
        return fr_unpack_chunks(self, payload, sums, chunk_ids, dst, bitmap, n_bad, stream, payload_bytes, sync)

    @property
    def delta_payload_max(self) -> int:
        return self.info["delta_payload_max"]

    def empty_delta_payload(self, device="cuda"):
        import torch

        return torch.empty(max(self.delta_payload_max, 16), dtype=torch.uint8, device=device)

    def pack_flagged(self, src, flagged, payload, sums, counts=None, stream=None, payload_cap=None):
        return fr_pack_flagged(self, src, flagged, payload, payload_cap, sums, counts, stream)

    def unpack_flagged(self, payload, sums, flagged, dst, bitmap, n_bad, stream=None, payload_bytes=None,
                       sync=False):
        return fr_unpack_flagged(self, payload, payload_bytes, sums, flagged, dst, bitmap, n_bad, stream, sync)


def _synced_bits(bitmap, n: int, stream) -> np.ndarray:
    """Wait for `stream` (None: the current stream; an int handle: the whole
    device), then return the sorted indices of the set bits of `bitmap`.
    The ``sync=True`` form of the operations that produce a bitmap."""
    import torch

    if n == 0:
        return np.zeros(0, dtype=np.int64)
    if not hasattr(bitmap, "detach"):
        raise ValueError("sync=True needs the bitmap as a tensor")
    if stream is None:
        torch.cuda.current_stream().synchronize()
    elif isinstance(stream, int):
        torch.cuda.synchronize()
    else:
        stream.synchronize()
    return bitmap_indices(bitmap, n)


def _nbytes(x):
    if x is None or isinstance(x, int):
        return None
    return x.numel() * x.element_size()


def fr_plan_create(table, chunk_bytes, src_arena_bytes, dst_arena_bytes) -> Plan:
    return Plan(table, chunk_bytes, src_arena_bytes, dst_arena_bytes)


def fr_plan_create_ex(table, chunk_bytes, src_arena_bytes, dst_arena_bytes, segment_align) -> Plan:
    return Plan(table, chunk_bytes, src_arena_bytes, dst_arena_bytes, segment_align)


def fr_plan_destroy(plan: Plan) -> None:
    plan.destroy()


def fr_pack_state(plan: Plan, src, payload, payload_cap, sums, stream=None) -> None:
    if payload_cap is None:
        payload_cap = _nbytes(payload)
        if payload_cap is None:
            payload_cap = plan.payload_bytes
    i = plan.info
    # pack writes payload_bytes (a smaller cap is the library's FR_E_RANGE)
    _check(_lib.fr_pack_state(plan.handle, _dev(src, i["src_arena_bytes"], "src"),
                              _dev(payload, min(payload_cap, i["payload_bytes"]), "payload"), payload_cap,
                              _dev(sums, SUM_BYTES * i["n_chunks"], "sums"), _stream(stream)),
           "fr_pack_state")


def fr_unpack_state(plan: Plan, payload, sums, dst, bad_bitmap, n_bad, stream=None, sync=False):
    """Enqueue the unpack; with sync=True wait for it and return the sorted
    ids of the chunks that failed verification (else None)."""
    i = plan.info
    _check(_lib.fr_unpack_state(plan.handle, _dev(payload, i["payload_bytes"], "payload"),
                                _dev(sums, SUM_BYTES * i["n_chunks"], "sums"),
                                _dev(dst, i["dst_arena_bytes"], "dst"),
                                _dev(bad_bitmap, 4 * i["bitmap_words"], "bad_bitmap"),
                                _dev(n_bad, 8, "n_bad"), _stream(stream)), "fr_unpack_state")
    return _synced_bits(bad_bitmap, i["n_chunks"], stream) if sync else None


def fr_verify_replicas(plan: Plan, base_a, base_b, diff_bitmap, n_diff, sums_a=None, sums_b=None,
                       stream=None, sync=False):
    """Enqueue the replica compare; with sync=True wait for it and return the
    sorted ids of the chunks that differ (else None)."""
    i = plan.info
    sb = SUM_BYTES * i["n_chunks"]
    _check(_lib.fr_verify_replicas(plan.handle, _dev(base_a, i["src_arena_bytes"], "base_a"),
                                   _dev(base_b, i["src_arena_bytes"], "base_b"),
                                   _dev(diff_bitmap, 4 * i["bitmap_words"], "diff_bitmap"),
                                   _dev(n_diff, 8, "n_diff"), _dev(sums_a, sb, "sums_a"),
                                   _dev(sums_b, sb, "sums_b"), _stream(stream)), "fr_verify_replicas")
    return _synced_bits(diff_bitmap, i["n_chunks"], stream) if sync else None


def fr_verify_replicas_noalloc(plan: Plan, base_a, base_b, diff_bitmap, n_diff, sums_a=None, sums_b=None,
                               stream=None, sync=False):
    """fr_verify_replicas with the library's static device scratch instead of
    the plan's (the call allocates nothing); same arguments and results."""
    i = plan.info
    sb = SUM_BYTES * i["n_chunks"]
    _check(_lib.fr_verify_replicas_noalloc(plan.handle, _dev(base_a, i["src_arena_bytes"], "base_a"),
                                           _dev(base_b, i["src_arena_bytes"], "base_b"),
                                           _dev(diff_bitmap, 4 * i["bitmap_words"], "diff_bitmap"),
                                           _dev(n_diff, 8, "n_diff"), _dev(sums_a, sb, "sums_a"),
                                           _dev(sums_b, sb, "sums_b"), _stream(stream)),
           "fr_verify_replicas_noalloc")
    return _synced_bits(diff_bitmap, i["n_chunks"], stream) if sync else None


def fr_compare_sums(plan: Plan, sums_a, sums_b, diff_bitmap, n_diff, stream=None, sync=False):
    """Enqueue the compare of two sums arrays (each from fr_checksum_state of
    one replica); with sync=True wait and return the sorted ids of the chunks
    whose sums differ (else None)."""
    i = plan.info
    sb = SUM_BYTES * i["n_chunks"]
    _check(_lib.fr_compare_sums(plan.handle, _dev(sums_a, sb, "sums_a"), _dev(sums_b, sb, "sums_b"),
                                _dev(diff_bitmap, 4 * i["bitmap_words"], "diff_bitmap"),
                                _dev(n_diff, 8, "n_diff"), _stream(stream)), "fr_compare_sums")
    return _synced_bits(diff_bitmap, i["n_chunks"], stream) if sync else None


def fr_checksum_state(plan: Plan, base, sums, stream=None) -> None:
    i = plan.info
    _check(_lib.fr_checksum_state(plan.handle, _dev(base, i["src_arena_bytes"], "base"),
                                  _dev(sums, SUM_BYTES * i["n_chunks"], "sums"), _stream(stream)),
           "fr_checksum_state")


def _ids(chunk_ids) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(chunk_ids, dtype=np.uint32).reshape(-1))


def fr_delta_layout(plan: Plan, chunk_ids) -> int:
    ids = _ids(chunk_ids)
    out = C.c_uint64()
    _check(_lib.fr_delta_layout(plan.handle, ids.ctypes.data if ids.size else None, ids.size,
                                C.byref(out)), "fr_delta_layout")
    return out.value


def fr_pack_chunks(plan: Plan, src, chunk_ids, payload, payload_cap, sums, stream=None) -> None:
    ids = _ids(chunk_ids)
    if payload_cap is None:
        payload_cap = _nbytes(payload)
        if payload_cap is None:
            payload_cap = fr_delta_layout(plan, ids)
    # the library refuses a cap below the list's payload and writes no more
    # than that, so a tensor of payload_cap bytes is enough
    _check(_lib.fr_pack_chunks(plan.handle, _dev(src, plan.info["src_arena_bytes"], "src"),
                               ids.ctypes.data if ids.size else None, ids.size,
                               _dev(payload, payload_cap, "payload"), payload_cap,
                               _dev(sums, SUM_BYTES * ids.size, "sums"), _stream(stream)), "fr_pack_chunks")


def fr_unpack_chunks(plan: Plan, payload, sums, chunk_ids, dst, bad_bitmap, n_bad, stream=None,
                     payload_bytes=None, sync=False):
    """payload_bytes: bytes readable at payload (default: the tensor's size,
    else the list's fr_delta_layout bytes); the library refuses less than the
    list needs.  With sync=True wait and return the sorted list positions
    that failed verification (else None)."""
    ids = _ids(chunk_ids)
    if payload_bytes is None:
        payload_bytes = _nbytes(payload)
        if payload_bytes is None:
            payload_bytes = fr_delta_layout(plan, ids)
    _check(_lib.fr_unpack_chunks(plan.handle, _dev(payload, payload_bytes, "payload"), payload_bytes,
                                 _dev(sums, SUM_BYTES * ids.size, "sums"),
                                 ids.ctypes.data if ids.size else None, ids.size,
                                 _dev(dst, plan.info["dst_arena_bytes"], "dst"),
                                 _dev(bad_bitmap, 4 * ((ids.size + 31) // 32), "bad_bitmap"),
                                 _dev(n_bad, 8, "n_bad"), _stream(stream)), "fr_unpack_chunks")
    return _synced_bits(bad_bitmap, ids.size, stream) if sync else None


class Tracker:
    """Step-tag tracker of the controller (``fr_tracker_*``; host only)."""

    def __init__(self, n_ranks: int, dp_group=None, timeout_s: float = 10.0, now_s: float = 0.0):
        self._h = None
        self.n_ranks = n_ranks
        g = None if dp_group is None else np.ascontiguousarray(dp_group, dtype=np.uint32).reshape(-1)
        if g is not None and g.size != n_ranks:
            raise ValueError(f"dp_group has {g.size} entries for {n_ranks} ranks")
        h = C.c_void_p()
        _check(_lib.fr_tracker_create(n_ranks, None if g is None else g.ctypes.data, timeout_s, now_s,
                                      C.byref(h)), "fr_tracker_create")
        self._h = h

    def __del__(self):
        if getattr(self, "_h", None) is not None:
            _lib.fr_tracker_destroy(self._h)
            self._h = None

    def heartbeat(self, rank: int, step_tag: int, now_s: float):
        _check(_lib.fr_tracker_heartbeat(self._h, rank, step_tag, now_s), "fr_tracker_heartbeat")

    def report_failure(self, rank: int, now_s: float):
        _check(_lib.fr_tracker_report_failure(self._h, rank, now_s), "fr_tracker_report_failure")

    def decide(self, now_s: float) -> dict:
        d = fr_decision()
        _check(_lib.fr_tracker_decide(self._h, now_s, C.byref(d)), "fr_tracker_decide")
        return {"action": ACTIONS[d.action], "resume_step": d.resume_step, "n_failed": d.n_failed,
                "n_waiting": d.n_waiting}

    def failed_ranks(self, now_s: float) -> list:
        out = np.zeros(self.n_ranks, np.uint32)
        n = C.c_uint32()
        _check(_lib.fr_tracker_failed_ranks(self._h, now_s, out.ctypes.data, self.n_ranks, C.byref(n)),
               "fr_tracker_failed_ranks")
        return [int(x) for x in out[: n.value]]

    def donors(self, now_s: float) -> list:
        out = np.zeros(self.n_ranks, np.int32)
        self.donors_into(now_s, out)
        return [int(x) for x in out]

    def donors_into(self, now_s: float, out: np.ndarray) -> np.ndarray:
        """donors() into a caller-owned contiguous int32 array of n_ranks."""
        if not (isinstance(out, np.ndarray) and out.dtype == np.int32 and out.size == self.n_ranks
                and out.flags.c_contiguous):
            raise ValueError("out must be a contiguous int32 array with one element per rank")
        _check(_lib.fr_tracker_donors(self._h, now_s, out.ctypes.data), "fr_tracker_donors")
        return out


class Layout3D:
    """A data x tensor x pipeline parallel layout with ZeRO sharding
    (``fr_layout_*``; host only)."""

    def __init__(self, tp=1, pp=1, dp=1, shard=1, zero_stage=0):
        self.s = fr_layout3d(tp, pp, dp, shard, zero_stage, 0)
        self.world = tp * pp * dp

    def coords(self, rank: int) -> tuple:
        out = np.zeros(5, np.uint32)
        _check(_lib.fr_layout_rank_coords(C.byref(self.s), rank, out.ctypes.data), "fr_layout_rank_coords")
        return tuple(int(x) for x in out)

    def donors(self, failed) -> list:
        f = np.zeros(self.world, np.uint8)
        f[list(failed)] = 1
        out = np.zeros(self.world, np.int32)
        return [int(x) for x in self.donors_into(f, out)]

    def donors_into(self, failed_mask: np.ndarray, out: np.ndarray) -> np.ndarray:
        """donors() from a uint8 mask of failed ranks into a caller-owned
        int32 array (both contiguous, one element per rank)."""
        for a, dt, name in ((failed_mask, np.uint8, "failed_mask"), (out, np.int32, "out")):
            if not (isinstance(a, np.ndarray) and a.dtype == dt and a.size == self.world and a.flags.c_contiguous):
                raise ValueError(f"{name} must be a contiguous {np.dtype(dt).name} array with one element per rank")
        _check(_lib.fr_layout_donors(C.byref(self.s), failed_mask.ctypes.data, out.ctypes.data),
               "fr_layout_donors")
        return out

    def state_table(self, rank: int, numel):
        """(table as a DESC_DTYPE array, arena bytes) of `rank`'s state."""
        n = np.ascontiguousarray(numel, np.uint64)
        ne, ab = C.c_uint32(), C.c_uint64()
        ptr = n.ctypes.data if n.size else None
        _check(_lib.fr_layout_state_table(C.byref(self.s), rank, ptr, n.size, None, 0, C.byref(ne), C.byref(ab)),
               "fr_layout_state_table")
        t = np.zeros(ne.value, DESC_DTYPE)
        _check(_lib.fr_layout_state_table(C.byref(self.s), rank, ptr, n.size, t.ctypes.data, ne.value,
                                          C.byref(ne), C.byref(ab)), "fr_layout_state_table")
        return t, ab.value


def fr_strerror(status: int) -> str:
    return _lib.fr_strerror(status).decode()


def fr_abi_version() -> int:
    return _lib.fr_abi_version()


def bitmap_indices(bitmap, n_chunks: int) -> np.ndarray:
    """Sorted chunk ids of the set bits of a result bitmap (host copy)."""
    b = bitmap.detach().cpu().numpy() if hasattr(bitmap, "detach") else np.asarray(bitmap)
    bits = np.unpackbits(np.ascontiguousarray(b).view(np.uint8), bitorder="little")
    return np.nonzero(bits[:n_chunks])[0]


def fr_pack_flagged(plan: Plan, src, flagged, payload, payload_cap, sums, counts=None, stream=None) -> None:
    """Delta pack of the chunks whose bits are set in the device bitmap
    `flagged`; `counts` (None or a device tensor of two int64) receives the
    list's length and its delta payload bytes."""
    i = plan.info
    if payload_cap is None:
        payload_cap = _nbytes(payload)
        if payload_cap is None:
            payload_cap = i["delta_payload_max"]
    _check(_lib.fr_pack_flagged(plan.handle, _dev(src, i["src_arena_bytes"], "src"),
                                _dev(flagged, 4 * i["bitmap_words"], "flagged"),
                                _dev(payload, min(payload_cap, i["delta_payload_max"]), "payload"), payload_cap,
                                _dev(sums, SUM_BYTES * i["n_chunks"], "sums"), _dev(counts, 16, "counts"),
                                _stream(stream)), "fr_pack_flagged")


def fr_unpack_flagged(plan: Plan, payload, payload_bytes, sums, flagged, dst, bad_bitmap, n_bad, stream=None,
                      sync=False):
    """Delta unpack of the chunks whose bits are set in `flagged`; with
    sync=True wait and return the sorted list positions that failed."""
    i = plan.info
    if payload_bytes is None:
        payload_bytes = _nbytes(payload)
        if payload_bytes is None:
            raise ValueError("payload_bytes is needed with a raw payload address")
    _check(_lib.fr_unpack_flagged(plan.handle, _dev(payload, payload_bytes, "payload"), payload_bytes,
                                  _dev(sums, SUM_BYTES * i["n_chunks"], "sums"),
                                  _dev(flagged, 4 * i["bitmap_words"], "flagged"),
                                  _dev(dst, i["dst_arena_bytes"], "dst"),
                                  _dev(bad_bitmap, 4 * i["bitmap_words"], "bad_bitmap"),
                                  _dev(n_bad, 8, "n_bad"), _stream(stream)), "fr_unpack_flagged")
    return _synced_bits(bad_bitmap, i["n_chunks"], stream) if sync else None
