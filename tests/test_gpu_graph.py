"""Streams and graphs.  A whole restore step captured in a HIP graph (the
operations are kernel launches only: no memsets, no host work on the stream)
and replayed several times, with eager work and synchronisation between
replays, every replay checked against the eager result; a replica compare and
the repair it drives (the flagged delta calls) captured and replayed on
different divergences; and two plans run concurrently on two streams."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402


def _scattered_case(C=4096):
    """40 tensors at shuffled 16-byte offsets (the same layout on both
    sides, so the receiver equals the sender): pack and unpack walk tiles."""
    rng = np.random.default_rng(8)
    t, sb, _ = W.random_tiny_table(rng, max_entries=40, max_numel=60_000)
    t["dst_offset"] = t["src_offset"]
    return t, C, sb, sb, W.random_tiny_state(t, sb, rng)


@pytest.mark.parametrize("case", ["toy", "scattered", "scattered 1 KiB chunks"])
def test_captured_restore_step_replays_correctly(case, monkeypatch):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if case == "toy":
        w = W.make_workload(0)
        table, C, sb, db, src_np = w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes, W.fill_state(w)
    else:  # 1 KiB chunks: unpack and the compare take 64 x 1 tiles, the checksum 64 x 4
        table, C, sb, db, src_np = _scattered_case(1024 if "1 KiB" in case else 4096)
    for k in [k for k in os.environ if k.startswith("FLASHRESTORE_TILE")]:
        monkeypatch.delenv(k)
    plan = F.Plan(table, C, sb, db)
    if case != "toy":
        assert plan.info["pack_walk"] == 4 and plan.info["unpack_walk"] == 4
    if "1 KiB" in case:
        assert (plan.info["tile_unpack"], plan.info["tile_verify"], plan.info["tile_checksum"]) == (7, 7, 4)
    src = torch.from_numpy(src_np).to("cuda")
    payload, sums = plan.empty_payload(), plan.empty_sums()
    dst = torch.zeros(db, dtype=torch.uint8, device="cuda")
    covered = torch.zeros(sb, dtype=torch.bool)  # the entries' bytes (the rest are gaps)
    plain = torch.zeros(sb, dtype=torch.bool)    # those of entries neither derived nor masters
    masters = {int(e["derive_from"]) for e in table if int(e["derive_from"]) >= 0}
    for k, e in enumerate(table):
        n = int(e["numel"]) * (4 if int(e["dtype"]) == F.FR_F32 else 2)
        covered[int(e["src_offset"]):int(e["src_offset"]) + n] = True
        if int(e["derive_from"]) < 0 and k not in masters:
            plain[int(e["src_offset"]):int(e["src_offset"]) + n] = True
    covered = covered.to("cuda")
    # flips go to plain entries: the receiver re-derives a derived entry from
    # its master, so a flip in either would (rightly) be flagged
    entries = torch.nonzero(plain).flatten().numpy()
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    csum = plan.empty_sums()

    def step():
        plan.pack(src, payload, sums)
        plan.unpack(payload, sums, dst, bad, nbad)
        plan.verify_replicas(src, dst, diff, ndiff)
        plan.checksum_state(dst, csum)

    # eager reference of the unmodified state
    step()
    torch.cuda.synchronize()
    assert torch.equal(dst[covered], src[covered]) and int(nbad.item()) == 0 and int(ndiff.item()) == 0
    ref = (payload.clone(), sums.clone(), dst.clone(), csum.clone())

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    rng = np.random.default_rng(3)
    for rep in range(4):
        # eager work between replays: perturb the donor, then restore it later
        flip = int(entries[int(rng.integers(0, entries.size))])
        src[flip] ^= 0x10
        dst.fill_(0x77)
        nbad.fill_(99)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        # the captured step saw the perturbed donor: check against eager
        exp_payload, exp_sums = plan.empty_payload(), plan.empty_sums()
        plan.pack(src, exp_payload, exp_sums)
        torch.cuda.synchronize()
        assert torch.equal(payload, exp_payload) and torch.equal(sums, exp_sums), rep
        assert torch.equal(dst[covered], src[covered]) and int(nbad.item()) == 0 and int(ndiff.item()) == 0
        assert torch.equal(csum, sums)
        src[flip] ^= 0x10  # undo
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(payload, ref[0]) and torch.equal(sums, ref[1])
    assert torch.equal(dst[covered], ref[2][covered]) and torch.equal(csum, ref[3])


def test_captured_compare_and_repair_replays_correctly():
    """Replica compare -> delta pack of the flagged chunks -> delta unpack
    into the replica, captured once and replayed on a different divergence
    each time: the replica equals the donor again, and the delta payload and
    sums equal the oracle's for the flagged list."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from oracle import cpu

    w = W.make_workload(0)
    t, C = w.table, w.chunk_bytes
    donor_np = W.fill_state(w)
    plan = F.Plan(t, C, w.src_arena_bytes, w.src_arena_bytes)
    donor = torch.from_numpy(donor_np).to("cuda")
    replica = donor.clone()
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    pay, sums = plan.empty_delta_payload(), plan.empty_sums()
    counts = torch.empty(2, dtype=torch.int64, device="cuda")
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()

    def repair():
        plan.verify_replicas(donor, replica, diff, ndiff)
        plan.pack_flagged(donor, diff, pay, sums, counts)
        plan.unpack_flagged(pay, sums, diff, replica, bad, nbad, payload_bytes=pay.numel())

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        repair()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        repair()
    torch.cuda.synchronize()

    rng = np.random.default_rng(17)
    for rep, k in enumerate((1, 7, 0, 300, 64)):
        pos = rng.choice(donor_np.size * 8, size=k, replace=False)
        rep_np = donor_np.copy()
        for p in pos:
            rep_np[p // 8] ^= np.uint8(1 << (p % 8))
        replica.copy_(torch.from_numpy(rep_np).to("cuda"))
        nbad.fill_(99)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        bm, nd = cpu.verify(t, C, donor_np, rep_np)
        ids = np.array(cpu.bitmap_to_set(bm, plan.n_chunks), np.uint32)
        opay, osums = cpu.pack_chunks(t, C, donor_np, ids)
        assert int(ndiff.item()) == nd and counts.tolist() == [ids.size, opay.size], rep
        assert np.array_equal(pay[: opay.size].cpu().numpy(), opay), rep
        assert np.array_equal(sums[: ids.size].cpu().numpy().view(np.uint64).reshape(-1), osums), rep
        assert int(nbad.item()) == 0 and torch.equal(replica, donor), rep


def test_captured_sums_check_and_repair_replays_correctly():
    """The cross-GPU form of the same repair, on one GPU: checksum of each
    replica -> fr_compare_sums of the two sums arrays -> delta pack of the
    flagged chunks -> delta unpack, captured once and replayed on a
    different divergence each time: the flagged set is the oracle's compare
    of the two replicas' sums, and the replica equals the donor again."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from oracle import cpu

    w = W.make_workload(0)
    t, C = w.table, w.chunk_bytes
    donor_np = W.fill_state(w)
    plan = F.Plan(t, C, w.src_arena_bytes, w.src_arena_bytes)
    donor = torch.from_numpy(donor_np).to("cuda")
    replica = donor.clone()
    sa, sb = plan.empty_sums(), plan.empty_sums()
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    pay, sums = plan.empty_delta_payload(), plan.empty_sums()
    counts = torch.empty(2, dtype=torch.int64, device="cuda")
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()

    def repair():
        plan.checksum_state(donor, sa)
        plan.checksum_state(replica, sb)
        plan.compare_sums(sa, sb, diff, ndiff)
        plan.pack_flagged(donor, diff, pay, sums, counts)
        plan.unpack_flagged(pay, sums, diff, replica, bad, nbad, payload_bytes=pay.numel())

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        repair()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        repair()
    torch.cuda.synchronize()

    rng = np.random.default_rng(23)
    ref = cpu.checksum(t, C, donor_np)
    for rep, k in enumerate((3, 0, 120, 1)):
        pos = rng.choice(donor_np.size * 8, size=k, replace=False)
        rep_np = donor_np.copy()
        for p in pos:
            rep_np[p // 8] ^= np.uint8(1 << (p % 8))
        replica.copy_(torch.from_numpy(rep_np).to("cuda"))
        nbad.fill_(99)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        bm, nd = cpu.compare_sums(ref, cpu.checksum(t, C, rep_np))
        ids = np.array(cpu.bitmap_to_set(bm, plan.n_chunks), np.uint32)
        assert int(ndiff.item()) == nd and int(counts[0].item()) == ids.size, rep
        assert int(nbad.item()) == 0 and torch.equal(replica, donor), rep


def test_two_plans_on_two_streams_run_concurrently():
    """One plan per concurrent stream: two plans' whole restore steps, queued
    on two streams without ordering between them, give the same results as
    each plan run alone."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(5)
    runs = []
    for seed in (0, 1):
        t, sb, db = W.random_tiny_table(rng, max_entries=40, max_numel=200_000)
        src = torch.from_numpy(W.random_tiny_state(t, sb, rng)).to("cuda")
        plan = F.Plan(t, 4096, sb, db)
        bufs = dict(payload=plan.empty_payload(), sums=plan.empty_sums(),
                    dst=torch.full((max(db, 1),), 0x5A, dtype=torch.uint8, device="cuda"),
                    bad=plan.empty_bitmap(), nbad=plan.empty_counter(), csum=plan.empty_sums())
        runs.append((plan, src, bufs))

    def step(plan, src, b, stream):
        plan.pack(src, b["payload"], b["sums"], stream=stream)
        plan.unpack(b["payload"], b["sums"], b["dst"], b["bad"], b["nbad"], stream=stream)
        plan.checksum_state(src, b["csum"], stream=stream)

    def view(plan, b):  # the bytes a step defines (the receiver's gaps keep their canary)
        return {"payload": b["payload"][: plan.payload_bytes], "sums": b["sums"][: plan.n_chunks],
                "dst": b["dst"], "bad": b["bad"], "nbad": b["nbad"], "csum": b["csum"][: plan.n_chunks]}

    # each alone, on the current stream
    ref = []
    for plan, src, b in runs:
        step(plan, src, b, torch.cuda.current_stream())
        torch.cuda.synchronize()
        ref.append({k: v.clone() for k, v in view(plan, b).items()})
        for k, v in b.items():
            v.fill_(0x5A if k == "dst" else 0x33)
    # both at once, on two streams
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for i in range(3):
        for (plan, src, b), s in zip(runs, streams):
            with torch.cuda.stream(s):
                step(plan, src, b, s)
    torch.cuda.synchronize()
    for (plan, src, b), r in zip(runs, ref):
        got = view(plan, b)
        for k in got:
            assert torch.equal(got[k], r[k]), k
        assert int(b["nbad"].item()) == 0


def test_two_plans_delta_calls_on_two_streams():
    """Delta calls of two plans (each with its own unit-record buffer) queued
    on two streams without ordering between them give each plan's serial
    results."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(6)
    runs = []
    for _ in range(2):
        t, sb, db = W.random_tiny_table(rng, max_entries=40, max_numel=200_000)
        src = torch.from_numpy(W.random_tiny_state(t, sb, rng)).to("cuda")
        plan = F.Plan(t, 4096, sb, db)
        n = plan.n_chunks
        ids = np.sort(rng.choice(n, size=max(1, n // 3), replace=False)).astype(np.uint32)
        pb = plan.delta_layout(ids)
        bufs = dict(payload=torch.full((max(pb, 16),), 0x33, dtype=torch.uint8, device="cuda"),
                    sums=torch.empty(ids.size, 2, dtype=torch.int64, device="cuda"),
                    dst=torch.full((max(db, 1),), 0x5A, dtype=torch.uint8, device="cuda"),
                    bad=torch.empty((ids.size + 31) // 32, dtype=torch.int32, device="cuda"),
                    nbad=plan.empty_counter())
        runs.append((plan, src, ids, pb, bufs))

    def step(plan, src, ids, b, stream):
        plan.pack_chunks(src, ids, b["payload"], b["sums"], stream=stream)
        plan.unpack_chunks(b["payload"], b["sums"], ids, b["dst"], b["bad"], b["nbad"], stream=stream)

    ref = []
    for plan, src, ids, pb, b in runs:
        step(plan, src, ids, b, torch.cuda.current_stream())
        torch.cuda.synchronize()
        # (the receiver starts as a canary arena, so a listed bf16 chunk whose
        # masters are not listed is re-derived from canary bytes and flagged;
        # the flags must match the serial run's)
        ref.append({"payload": b["payload"][:pb].clone(), "sums": b["sums"].clone(), "dst": b["dst"].clone(),
                    "bad": b["bad"].clone(), "nbad": b["nbad"].clone()})
        b["payload"].fill_(0x33)
        b["dst"].fill_(0x5A)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for _ in range(3):
        for (plan, src, ids, pb, b), s in zip(runs, streams):
            with torch.cuda.stream(s):
                step(plan, src, ids, b, s)
    torch.cuda.synchronize()
    for (plan, src, ids, pb, b), r in zip(runs, ref):
        assert torch.equal(b["payload"][:pb], r["payload"]) and torch.equal(b["sums"], r["sums"])
        assert torch.equal(b["dst"], r["dst"])
        assert torch.equal(b["bad"], r["bad"]) and torch.equal(b["nbad"], r["nbad"])
