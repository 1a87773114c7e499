#!/usr/bin/env python3
"""Benchmark of the replica state-restore hot path on one MI355X.

One step = one pass of the whole path over one rank's training state:
  pack + checksum (donor) -> unpack + bf16 re-derive + verify (receiver)
  -> replica compare (donor vs restored) -> checksum of the restored state.
(When the receiver's layout differs from the donor's, as in the descriptor
stress workload, the compare and the checksum take a second replica in the
donor's layout instead of the restored arena.)
The workload is one rank's share of a Llama-3-8B-shaped state under tensor
parallel 8 (1,004,015,616 params; bf16 param + fp32 master + fp32 Adam m, v =
14,056,218,624 bytes; 64 KiB chunks), synthetic values, resident in HBM
before timing starts.  The plan (descriptor validation and device tables) is
built once, outside the timed region.

Prints one JSON line.  `value` is the restore rate the metric names: state
bytes over the time of pack + checksum and unpack + verify (the two
operations of a restore); `step_gbs` is the state over the whole step's
time.  Also: per-operation times, algorithmic HBM GB/s, fractions of the HBM
peak and of the copy / read-only ceilings measured in the same process with
plain streaming kernels, a roofline entry for the dominant kernel, and the
CPU oracle's rates on a stated sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
METRIC = "state restore GB/s per GPU (pack+checksum, unpack+verify) and % of HBM peak"
KERNEL_SOURCES = ("paper_2509_03047_amd/csrc/kernels.hip", "paper_2509_03047_amd/csrc/fr_internal.h")
# HBM traffic per launch measured with rocprofv3 counters, per workload
TRAFFIC_FILES = {1: "hbm_traffic_llama8b_tp8.json", 2: "hbm_traffic_descriptor_stress_20k.json",
                 3: "hbm_traffic_llama70b_tp8pp4.json"}
KERNEL_NAMES = {"pack": "k_pack", "unpack": "k_unpack", "verify": "k_verify", "checksum": "k_pack"}
WALK_TILES = 4  # fr_plan_info pack_walk / unpack_walk: one aligned tile of the side written per workgroup
TILE_KERNELS = {"pack": "k_pack_blocks", "unpack": "k_unpack_blocks"}
WALK_NAMES = {0: "slices", 1: "slices cut at arena / receiver lines", 2: "slices cut at payload lines",
              3: "slices cut at payload slice boundaries", WALK_TILES: "tiles of the side written"}
# fr_plan_info tile_*: threads x 16-byte vectors per workgroup
TILE_SHAPES = ("256x1", "512x1", "256x2", "256x4", "64x4", "128x2", "64x2", "64x1", "128x1", "128x4", "64x8")


def _code_only(text: str) -> str:
    """C++ source without comments and with whitespace collapsed, so that a
    comment edit does not count as a kernel change (string literals in these
    sources hold no comment markers)."""
    import re

    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(read=None) -> str:
    """Hash of the kernel sources' code (comments excluded); `read(path)`
    supplies a file's text (default: the working tree)."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        if read is None:
            with open(os.path.join(ROOT, p), encoding="utf-8") as f:
                text = f.read()
        else:
            text = read(p)
        h.update(_code_only(text).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=1, help="workload: 0 toy, 1 8B share, 2 stress, 3 70B share")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-delta", action="store_true", help="skip the delta-repair measurement")
    ap.add_argument("--delta-flips", type=int, default=4096)
    ap.add_argument("--segment-align", type=int, default=None,
                    help="payload segment alignment (default: the library's, 16)")
    ap.add_argument("--cpu-sample-bytes", type=int, default=4_200_000_000,
                    help="state bytes of the oracle's sample (a prefix of the table)")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the copy / read ceiling kernels")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 4 GiB device copy (for counter scaling) and exit")
    return ap.parse_args()


def segment_bytes(table) -> int:
    """Bytes of the payload's segments: every sent (non-derived) entry padded
    to 16 bytes; the zero gaps between segments are not counted."""
    import numpy as np

    sent = table["derive_from"] < 0
    nb = table["numel"].astype(np.uint64) * np.where(table["dtype"] == 1, 4, 2).astype(np.uint64)
    return int(((nb[sent] + 15) // 16 * 16).sum())


def algorithmic_bytes(info, table=None) -> dict:
    """Bytes each operation must move at least (read + write), per launch.
    Pack writes the whole payload, zero gaps included; unpack reads only its
    segments (the whole payload when no table is given)."""
    S, P, n = info["state_bytes"], info["payload_bytes"], info["n_chunks"]
    R = P if table is None else segment_bytes(table)
    words = info["bitmap_words"]
    return {
        "pack": S + P + 16 * n,
        "unpack": R + 16 * n + S + 4 * words,
        "verify": 2 * S + 4 * words,
        "checksum": S + 16 * n,
    }


def copy_calibration():
    """Known traffic for scaling the HBM counters: a 4 GiB device copy
    (torch's, the runtime's copy kernel) ten times after five warm-ups, then
    one launch each of the plain copy and read-only kernels of libfrceil on
    the same 4 GiB (reads 4 GiB and writes 4 GiB; reads 4 GiB)."""
    import ctypes

    import torch

    from paper_2509_03047_amd import build as B

    n = 4 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    reps = 10
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    lib = ctypes.CDLL(B.CEIL_LIB)
    P, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
    lib.frc_copy.argtypes = [P, P, u64, P]
    lib.frc_read.argtypes = [P, u64, u32, P, P]
    sink = torch.zeros(64, dtype=torch.int32, device="cuda")
    sp = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if lib.frc_copy(b.data_ptr(), a.data_ptr(), n, sp) or lib.frc_read(a.data_ptr(), n, 7, sink.data_ptr(), sp):
        raise RuntimeError("ceiling kernel launch failed")
    torch.cuda.synchronize()
    return {"bytes_per_copy": 2 * n, "ms": ms, "gbs": 2 * n / ms / 1e6,
            "plain_kernels": {"k_copy": {"read": n, "write": n}, "k_read": {"read": n, "write": 0}}}


def ceilings(reps: int = 10, nbytes: int = 4 << 30):
    """Copy, read-only and write-only rates of plain streaming kernels on
    this GPU (libfrceil: 16-byte non-temporal accesses, 64-lane workgroups in
    address order, 1 KiB per workgroup for the copy and 4 KiB for the
    others): median GB/s over `reps` launches of `nbytes` each (a copy counts
    its reads and writes), timed with HIP events on the launch stream."""
    import ctypes

    import torch

    from paper_2509_03047_amd import build as B

    lib = ctypes.CDLL(B.CEIL_LIB)
    P, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
    lib.frc_copy.argtypes = [P, P, u64, P]
    lib.frc_read.argtypes = [P, u64, u32, P, P]
    lib.frc_write.argtypes = [P, u64, u32, P]
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(64, dtype=torch.int32, device="cuda")
    a.fill_(0x5A)
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    # the XOR of 16 words of 0x5A5A5A5A is 0, so 1 never occurs
    runs = {
        "copy": (2 * nbytes, lambda: lib.frc_copy(b.data_ptr(), a.data_ptr(), nbytes, sp)),
        "read": (nbytes, lambda: lib.frc_read(a.data_ptr(), nbytes, 1, sink.data_ptr(), sp)),
        "write": (nbytes, lambda: lib.frc_write(b.data_ptr(), nbytes, 7, sp)),
    }
    out = {}
    for name, (moved, fn) in runs.items():
        ts = []
        for i in range(reps + 3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = fn()
            e1.record(stream)
            if rc != 0:
                raise RuntimeError(f"ceiling kernel {name}: HIP error {rc}")
            torch.cuda.synchronize()
            if i >= 3:
                ts.append(e0.elapsed_time(e1))
        out[name + "_gbs"] = round(moved / (statistics.median(ts) * 1e-3) / 1e9, 1)
    if int(sink.abs().sum().item()) != 0:
        raise RuntimeError("read ceiling: the sink was written")
    del a, b
    torch.cuda.empty_cache()
    out["bytes"] = nbytes
    return out


# the ceiling each operation's traffic mix is measured against
CEILING_OF = {"pack": "copy", "unpack": "copy", "verify": "read", "checksum": "read"}


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_sample(w, src_np, max_bytes: int):
    """The first entries of the table (whole logical tensors for the
    model-shaped ones) up to about max_bytes of state, with the arenas the
    oracle reads and writes for them."""
    import numpy as np

    t = w.table
    es = np.where(t["dtype"] == 1, 4, 2).astype(np.int64) * t["numel"].astype(np.int64)
    cum = np.cumsum(es)
    step = 4 if w.tensors is not None else 1  # 4 entries per logical tensor
    n_ent = step
    while n_ent + step <= len(t) and cum[n_ent + step - 1] <= max_bytes:
        n_ent += step
    sub = t[:n_ent].copy()
    same_layout = (w.src_arena_bytes == w.dst_arena_bytes
                   and np.array_equal(t["src_offset"], t["dst_offset"]))
    if same_layout and w.tensors is not None:
        # entries are contiguous from 0: only the prefix's bytes are needed
        end = int(sub["src_offset"][-1]) + int(es[n_ent - 1])
        src, dst = src_np[:end], np.empty(end, np.uint8)
    else:
        src, dst = src_np, np.empty(w.dst_arena_bytes, np.uint8)
    # the compare and the checksum take an arena in the donor's layout
    replica = dst if same_layout else src
    what = f"{n_ent // 4} logical tensors" if step == 4 else "entries in table order"
    return sub, int(cum[n_ent - 1]), src, dst, replica, f"first {n_ent} of {len(t)} entries ({what}"


def _oracle_ops(sub, C, src, dst, replica, reps: int):
    """`reps` full oracle steps; per operation the median seconds."""
    import numpy as np

    from oracle import cpu

    ops = {"pack": [], "unpack": [], "verify": [], "checksum": []}
    for _ in range(reps):
        a = time.perf_counter()
        pay, sums = cpu.pack(sub, C, src)
        b = time.perf_counter()
        bm, nbad = cpu.unpack(sub, C, pay, sums, dst)
        c = time.perf_counter()
        vb, nd = cpu.verify(sub, C, src, replica)
        d = time.perf_counter()
        cs = cpu.checksum(sub, C, replica)
        e = time.perf_counter()
        for k, dt in zip(ops, (b - a, c - b, d - c, e - d)):
            ops[k].append(dt)
        if not (nbad == 0 and nd == 0 and np.array_equal(cs, sums)):
            raise RuntimeError("the oracle's own restore of the sample is not exact")
    return {k: statistics.median(v) for k, v in ops.items()}


def cpu_baseline(w, src_np, max_bytes: int = 4_200_000_000, reps: int = 3):
    """The oracle, as it stands, on a prefix of the same workload: the first
    entries of the table (the embedding and the first layers for the
    model-shaped ones) up to about `max_bytes` of state, on every host
    thread and on one thread.  Each operation's time is the median of
    `reps` full steps.  `value` is the restore rate in the unit of the
    benchmark's value: sample state bytes over the median pack plus the
    median unpack time; `ops_gbs` are state bytes per second of each
    operation alone."""
    from oracle import cpu

    C = w.chunk_bytes
    cores = cpu.threads()
    sub, state, src, dst, replica, what = _oracle_sample(w, src_np, max_bytes)

    def rates(med):
        return {"value": round(state / (med["pack"] + med["unpack"]) / 1e9, 4),
                "ops_gbs": {k: round(state / v / 1e9, 4) for k, v in med.items()},
                "ops_s": {k: round(v, 4) for k, v in med.items()}}

    t0 = time.perf_counter()
    many = rates(_oracle_ops(sub, C, src, dst, replica, reps))
    cpu.set_threads(1)
    try:
        one = rates(_oracle_ops(sub, C, src, dst, replica, reps))
    finally:
        cpu.set_threads(cores)
    pct = 100.0 * state / w.state_bytes
    return {
        "value": many["value"],
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{what}, {state} state bytes = {pct:.1f} % of the workload's {w.state_bytes}); "
                  f"median of {reps} full steps (pack+unpack+verify+checksum) per operation, "
                  f"value = sample bytes / (pack + unpack); {time.perf_counter() - t0:.1f} s in all",
        "ops_gbs": many["ops_gbs"],
        "ops_s": many["ops_s"],
        "cpu_model": _cpu_model(),
        "one_thread": {"value": one["value"], "unit": "GB/s", "cores": 1, "ops_gbs": one["ops_gbs"],
                       "ops_s": one["ops_s"], "sample": "the same"},
    }


def control_plane(reps=21):
    """Host rows at the paper's cluster scale, 4,800 ranks (TP 8 x PP 4 x
    DP 150, a 70B-class layout): step-tag tracker and restore planner
    latencies through the Python binding (medians; microseconds).  The 8
    ranks of one node fail in forward of step 41; every normal rank then
    reports 41."""
    import numpy as np

    from paper_2509_03047_amd import flashrestore as F
    from paper_2509_03047_amd import workloads as W

    tp, pp, dp = 8, 4, 150
    layout = F.Layout3D(tp, pp, dp, 1, 0)
    world = layout.world
    group = [c[1] * tp + c[0] for c in (layout.coords(r) for r in range(world))]
    failed = list(range(8 * 37, 8 * 38))  # one tensor-parallel group: a node
    failed_set = set(failed)

    def med_us(fn):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return round(statistics.median(ts) * 1e6, 1)

    tr = F.Tracker(world, group, 10.0, 0.0)
    t0 = time.perf_counter()
    for r in range(world):
        tr.heartbeat(r, 41, 1.0)
    hb_us = (time.perf_counter() - t0) / world * 1e6
    for r in failed:
        tr.report_failure(r, 2.0)
    for r in range(world):
        if r not in failed_set:
            tr.heartbeat(r, 41, 3.0)
    d = tr.decide(3.5)
    donors = tr.donors(3.5)
    ok = (d["action"] == "stop_and_restore" and d["resume_step"] == 41
          and all(donors[r] >= 0 and group[donors[r]] == group[r] for r in failed))
    numel = [n for _, n in W.llama3_70b_tp8_pp4_stage0_tensors()]
    zero1 = F.Layout3D(tp, pp, dp, 6, 1)
    out = np.zeros(world, np.int32)
    mask = np.zeros(world, np.uint8)
    mask[failed] = 1
    return {
        "ranks": world,
        "layout": "tp8 x pp4 x dp150",
        "tracker_heartbeat_us": round(hb_us, 2),
        "tracker_decide_us": med_us(lambda: tr.decide(3.5)),
        "tracker_donors_us": med_us(lambda: tr.donors_into(3.5, out)),
        "planner_donors_us": med_us(lambda: layout.donors_into(mask, out)),
        "planner_state_table_us": med_us(lambda: layout.state_table(failed[0], numel)),
        "planner_state_table_zero1_us": med_us(lambda: zero1.state_table(failed[0], numel)),
        "ok": bool(ok),
    }


def flips(table, C, k):
    """k distinct random bit flips over the table-order concatenation of the
    tensors' bytes (seed 4000 + k), mapped to arena offsets: (byte indices,
    XOR masks) as device tensors, and the set of chunks they fall in."""
    import numpy as np
    import torch

    from paper_2509_03047_amd import workloads as W

    nb = table["numel"].astype(np.int64) * np.where(table["dtype"] == W.F32, 4, 2)
    starts = np.concatenate([[0], np.cumsum(nb)])
    nch = -(-nb // C)
    base = np.concatenate([[0], np.cumsum(nch)])
    pos = W.flip_positions(int(starts[-1]) * 8, k, 4000 + k).astype(np.int64)
    cat = pos // 8
    e = np.searchsorted(starts, cat, side="right") - 1
    chunks = set(int(x) for x in base[e] + (cat - starts[e]) // C)
    by = table["src_offset"].astype(np.int64)[e] + (cat - starts[e])
    order = np.argsort(by, kind="stable")
    by, pos = by[order], pos[order]
    masks = (np.uint8(1) << (pos % 8).astype(np.uint8)).astype(np.uint8)
    uniq, start = np.unique(by, return_index=True)
    idx = torch.from_numpy(uniq).to("cuda")
    xor = torch.from_numpy(np.bitwise_or.reduceat(masks, start)).to("cuda")
    return idx, xor, chunks


def replica_compare(plan, table, donor, replica, stream, ks=(0, 1, 64, 4096), reps=5):
    """The replica compare on two copies of the state with k distinct random
    bit flips in the second: median time (HIP events) and whether the flagged
    set is exactly {chunk of each flipped byte}; and the same from the two
    copies' chunk sums alone (fr_compare_sums, the check replicas on
    different GPUs run after exchanging their sums): its median time and
    whether its set is the same.  The copy is restored after each k by
    flipping the same bits back."""
    import numpy as np
    import torch

    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    sums_a, sums_b = plan.empty_sums(), plan.empty_sums()
    plan.checksum_state(donor, sums_a, stream=stream)
    out = {}
    for k in ks:
        idx, xor, expect = flips(table, plan.info["chunk_bytes"], k)
        replica[idx] ^= xor
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            plan.verify_replicas(donor, replica, diff, ndiff, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        got = plan.verify_replicas(donor, replica, diff, ndiff, stream=stream, sync=True)
        n_diff = int(ndiff.item())
        plan.checksum_state(replica, sums_b, stream=stream)
        ss = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            plan.compare_sums(sums_a, sums_b, diff, ndiff, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ss.append(e0.elapsed_time(e1))
        got_s = plan.compare_sums(sums_a, sums_b, diff, ndiff, stream=stream, sync=True)
        replica[idx] ^= xor
        out[str(k)] = {"ms": round(float(np.median(ts)), 4), "n_diff": n_diff,
                       "exact": set(int(x) for x in got) == expect,
                       "sums_ms": round(float(np.median(ss)), 4),
                       "sums_exact": set(int(x) for x in got_s) == expect}
    torch.cuda.synchronize()
    return out


def delta_repair(plan, table, donor, replica, k, stream, reps=5):
    """Repair of a replica that diverged in k random bits of its tensors.
    Device-resident: compare, then the delta pack and unpack driven by the
    compare's bitmap (the list and its layout built on the device), all
    stream-ordered with no host round trip; timed with HIP events (compare,
    repair) and on the host clock from the compare's launch to the repaired
    replica.  For comparison, the repair through a host list (the flagged set
    read back, the list passed to the host-list calls).  `plan` has the
    donor's layout on both sides (replicas of one group share it)."""
    import numpy as np
    import torch

    from paper_2509_03047_amd import flashrestore as F

    idx, xor, expect = flips(table, plan.info["chunk_bytes"], k)
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    pay, sums = plan.empty_delta_payload(), plan.empty_sums()
    counts = torch.empty(2, dtype=torch.int64, device="cuda")

    def ev():
        return torch.cuda.Event(enable_timing=True)

    cmp_ms, rep_ms, wall_ms, over_ms = [], [], [], []
    ok = True
    for _ in range(reps):
        replica[idx] = replica[idx] ^ xor  # diverge
        torch.cuda.synchronize()
        e0, e1, e2 = ev(), ev(), ev()
        t0 = time.perf_counter()
        e0.record(stream)
        plan.verify_replicas(donor, replica, diff, ndiff, stream=stream)
        e1.record(stream)
        plan.pack_flagged(donor, diff, pay, sums, counts, stream=stream)
        plan.unpack_flagged(pay, sums, diff, replica, bad, nbad, stream=stream, payload_bytes=pay.numel())
        e2.record(stream)
        stream.synchronize()
        wall = (time.perf_counter() - t0) * 1e3
        cmp_ms.append(e0.elapsed_time(e1))
        rep_ms.append(e1.elapsed_time(e2))
        wall_ms.append(wall)
        over_ms.append(wall - e0.elapsed_time(e1))
        ok = ok and int(nbad.item()) == 0 and int(ndiff.item()) == len(expect)
    ok = ok and torch.equal(replica, donor)
    n_ids, pbytes = (int(x) for x in counts.tolist())

    # the same repair through a host list
    payload = torch.empty(max(pbytes, 16), dtype=torch.uint8, device="cuda")
    lsums = plan.empty_sums()
    list_gpu, list_wall = [], []
    for _ in range(reps):
        replica[idx] = replica[idx] ^ xor
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        plan.verify_replicas(donor, replica, diff, ndiff, stream=stream)
        ids = F.bitmap_indices(diff, plan.n_chunks).astype(np.uint32)  # synchronises
        e0, e1 = ev(), ev()
        e0.record(stream)
        plan.pack_chunks(donor, ids, payload, lsums, stream=stream)
        plan.unpack_chunks(payload, lsums, ids, replica, bad, nbad, stream=stream)
        e1.record(stream)
        stream.synchronize()
        list_wall.append((time.perf_counter() - t0) * 1e3)
        list_gpu.append(e0.elapsed_time(e1))
        ok = ok and int(nbad.item()) == 0 and ids.size == n_ids
    ok = ok and torch.equal(replica, donor)
    med = lambda v: round(float(np.median(v)), 4)  # noqa: E731
    return {
        "flips": k,
        "chunks_resent": n_ids,
        "payload_bytes": pbytes,
        "gpu_ms_compare": med(cmp_ms),
        "gpu_ms_repair": med(rep_ms),
        "wall_ms_compare_to_repaired": med(wall_ms),
        "wall_ms_beyond_compare": med(over_ms),
        "host_list": {"gpu_ms_pack_unpack": med(list_gpu), "wall_ms_compare_to_repaired": med(list_wall)},
        "full_restore_ms": None,
        "ok": bool(ok),
    }


def restored_equals(w, src, dst, batch_bytes: int = 1 << 26) -> bool:
    """Every entry's bytes at its receiver offset equal the donor's.  Entries
    are compared in batches of about `batch_bytes`: one gather of the batch's
    bytes from each arena (index ranges built on the device) and one compare,
    rather than a compare and a host synchronisation per entry."""
    import numpy as np
    import torch

    from paper_2509_03047_amd import workloads as W

    t = w.table
    nb = t["numel"].astype(np.int64) * np.where(t["dtype"] == W.F32, 4, 2)
    keep = nb > 0
    so, do, nb = t["src_offset"][keep].astype(np.int64), t["dst_offset"][keep].astype(np.int64), nb[keep]
    ends = np.cumsum(nb)
    ok = torch.ones((), dtype=torch.bool, device=src.device)
    first = 0
    while first < nb.size:
        last = int(np.searchsorted(ends, ends[first] - nb[first] + batch_bytes, side="right"))
        last = max(last, first + 1)
        lens = torch.from_numpy(nb[first:last]).to(src.device)
        pos = torch.arange(int(lens.sum()), device=src.device)
        base = torch.repeat_interleave(torch.cumsum(lens, 0) - lens, lens)
        off = pos - base  # byte within its entry
        i_src = torch.repeat_interleave(torch.from_numpy(so[first:last]).to(src.device), lens) + off
        i_dst = torch.repeat_interleave(torch.from_numpy(do[first:last]).to(src.device), lens) + off
        ok &= (src[i_src] == dst[i_dst]).all()
        first = last
    return bool(ok.item())


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU transport "
              "(a restore shards per rank: each GPU packs or unpacks its own share). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        print(json.dumps({"copy_calibration": copy_calibration()}), flush=True)
        return

    from paper_2509_03047_amd import flashrestore as F
    from paper_2509_03047_amd import workloads as W

    w = W.make_workload(args.config)
    t0 = time.perf_counter()
    src_np = W.fill_state(w)
    print(f"# generated {w.name}: {w.state_bytes} state bytes in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)
    torch.zeros(1, device="cuda")  # HIP runtime set-up, which the first plan would otherwise pay
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    plan = F.Plan(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes, args.segment_align)
    plan_ms = (time.perf_counter() - t0) * 1e3  # validation, walks, device tables (once per rank)
    info = plan.info
    src = torch.from_numpy(src_np).to("cuda")
    payload, sums = plan.empty_payload(), plan.empty_sums()
    dst = torch.empty(w.dst_arena_bytes, dtype=torch.uint8, device="cuda")
    same_layout = (w.src_arena_bytes == w.dst_arena_bytes
                   and np.array_equal(w.table["src_offset"], w.table["dst_offset"]))
    # arena compared with the donor and checksummed: the restored one, or a
    # second replica in the donor's layout
    replica = dst if same_layout else src.clone()
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    csum = plan.empty_sums()
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    ops = ("pack", "unpack", "verify", "checksum")

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        plan.pack(src, payload, sums, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        plan.unpack(payload, sums, dst, bad, nbad, stream=stream)
        if ev is not None:
            ev[2].record(stream)
        plan.verify_replicas(src, replica, diff, ndiff, stream=stream)
        if ev is not None:
            ev[3].record(stream)
        plan.checksum_state(replica, csum, stream=stream)
        if ev is not None:
            ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for k in range(args.steps):
        step(evs[k])
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)
    op_ms = {op: [e[i].elapsed_time(e[i + 1]) for e in evs] for i, op in enumerate(ops)}
    per_op = {op: sum(v) / len(v) for op, v in op_ms.items()}

    # the pass restored the state exactly: nothing flagged, receiver == sender
    ok = int(nbad.item()) == 0 and int(ndiff.item()) == 0
    ok = ok and torch.equal(csum[: plan.n_chunks], sums[: plan.n_chunks])
    ok = ok and (torch.equal(dst, src) if same_layout else restored_equals(w, src, dst))

    ms_step = total_ms / args.steps
    restore_ms = per_op["pack"] + per_op["unpack"]
    value = info["state_bytes"] / (restore_ms * 1e-3) / 1e9  # the metric: pack + unpack
    alg = algorithmic_bytes(info, w.table)
    op_report = {}
    for op in ops:
        gbs = alg[op] / (per_op[op] * 1e-3) / 1e9
        op_report[op] = {"ms": round(per_op[op], 4), "ms_median": round(statistics.median(op_ms[op]), 4),
                         "ms_min": round(min(op_ms[op]), 4), "alg_bytes": alg[op],
                         "hbm_gbs": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}
    dom = max(ops, key=lambda o: per_op[o])
    walks = {"pack": info["pack_walk"], "unpack": info["unpack_walk"]}
    kernel = TILE_KERNELS[dom] if walks.get(dom) == WALK_TILES else KERNEL_NAMES[dom]
    roof = {"bound": "hbm", "kernel": kernel, "op": dom,
            "achieved": op_report[dom]["hbm_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": op_report[dom]["frac_of_peak"], "traffic": None}
    try:  # counters taken on these kernels' code for this workload, else null
        with open(os.path.join(ROOT, "profiles", TRAFFIC_FILES[args.config])) as f:
            tr = json.load(f)
        if (tr.get("kernel_source_sha") == kernel_source_hash() and tr.get("config") == args.config
                and args.segment_align in (None, 16)):
            roof["traffic"] = tr.get("ops", {}).get(dom, {}).get("bytes_per_launch")
    except (KeyError, OSError, ValueError):
        pass

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32/u64",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "params": w.n_params,
            "state_bytes": info["state_bytes"],
            "payload_bytes": info["payload_bytes"],
            "chunk_bytes": info["chunk_bytes"],
            "segment_align": info["segment_align"],
            "n_chunks": info["n_chunks"],
            "step": "pack+checksum -> unpack+derive+verify -> verify_replicas -> checksum_state",
            "walks": {op: WALK_NAMES.get(v, str(v)) for op, v in walks.items()},
            "tiles": {op: TILE_SHAPES[info[f"tile_{op}"]] if info[f"tile_{op}"] < len(TILE_SHAPES)
                      else str(info[f"tile_{op}"]) for op in ("pack", "unpack", "verify", "checksum")},
        },
        "restore_ms": round(restore_ms, 4),
        "step_gbs": round(info["state_bytes"] / (ms_step * 1e-3) / 1e9, 2),
        "plan_ms": round(plan_ms, 2),
        "ops": op_report,
        "roofline": roof,
        "parity_ok": bool(ok),
        "wall_s_timed": round(wall, 4),
    }
    if not args.no_delta:
        rplan, rtable = plan, w.table
        if not same_layout:  # repair within the donor's layout
            rtable = w.table.copy()
            rtable["dst_offset"] = rtable["src_offset"]
            rplan = F.Plan(rtable, w.chunk_bytes, w.src_arena_bytes, w.src_arena_bytes, args.segment_align)
        out["replica_compare"] = replica_compare(rplan, rtable, src, replica, stream)
        out["delta_repair"] = delta_repair(rplan, rtable, src, replica, args.delta_flips, stream)
        out["delta_repair"]["full_restore_ms"] = round(restore_ms, 4)
    if not args.no_ceilings:
        ceil = ceilings()
        out["ceilings"] = ceil
        for op in ops:
            c = ceil[CEILING_OF[op] + "_gbs"]
            out["ops"][op]["ceiling"] = CEILING_OF[op]
            out["ops"][op]["frac_of_ceiling"] = round(out["ops"][op]["hbm_gbs"] / c, 4)
    out["control_plane"] = control_plane()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, src_np, args.cpu_sample_bytes)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
