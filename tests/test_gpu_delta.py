"""GPU parity of delta repair (re-sending only the diverged chunks) against the
CPU oracle, through the C ABI: payload, sums, receiver arena and result sets
bit for bit on random tables and lists, every tile, and a full-size repair of
the Llama-3-8B TP=8 rank share from the chunks the replica compare flags."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests.gpu_util import log, sums_host, to_dev, to_host  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def flagged_bitmap(plan, ids):
    """The device bitmap over the plan's chunk ids with the bits of `ids` set."""
    bits = np.zeros(max(plan.bitmap_words, 1), np.uint32)
    np.bitwise_or.at(bits, ids.astype(np.int64) >> 5, (np.uint32(1) << (ids & 31).astype(np.uint32)))
    return to_dev(bits.view(np.int32))


def _one(t, C, src_np, recv_np, ids, rng, tag, seg=None):
    """The host-list calls and the bitmap-driven calls on one list, each
    against the oracle: delta payload (gaps included), sums, receiver arena
    and result set, with the wire corrupted at random."""
    plan = F.Plan(t, C, max(src_np.size, 16), max(recv_np.size, 16), seg)
    oseg = cpu.SEGMENT if seg is None else seg
    src = to_dev(src_np) if src_np.size else torch.zeros(16, dtype=torch.uint8, device="cuda")
    dst = to_dev(recv_np) if recv_np.size else torch.zeros(16, dtype=torch.uint8, device="cuda")
    dst2 = dst.clone()
    pb = plan.delta_layout(ids)
    off, opb = cpu.delta_layout(t, C, ids, oseg)
    assert pb == opb, tag
    assert pb <= plan.delta_payload_max, tag
    payload = torch.full((max(pb, 16),), 0xEE, dtype=torch.uint8, device="cuda")  # gaps must be written
    sums = torch.empty(max(ids.size, 1), 2, dtype=torch.int64, device="cuda")
    plan.pack_chunks(src, ids, payload, sums)
    opay, osums = cpu.pack_chunks(t, C, src_np, ids, oseg)
    flagged = flagged_bitmap(plan, ids)
    fpay = plan.empty_delta_payload().fill_(0xEE)
    fsums = plan.empty_sums().fill_(-1)
    counts = torch.full((2,), -1, dtype=torch.int64, device="cuda")
    plan.pack_flagged(src, flagged, fpay, fsums, counts)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(payload)[:pb], opay), f"payload {tag}"
    assert np.array_equal(sums_host(sums, ids.size), osums), f"sums {tag}"
    assert counts.tolist() == [ids.size, pb], f"flagged counts {tag}"
    assert np.array_equal(to_host(fpay)[:pb], opay), f"flagged payload {tag}"
    assert np.array_equal(sums_host(fsums, ids.size), osums), f"flagged sums {tag}"
    assert bool((fsums[ids.size:] == -1).all()), f"flagged sums past the list {tag}"
    if pb and rng.random() < 0.4:  # corrupt the wire
        b = int(rng.integers(0, pb * 8))
        opay[b // 8] ^= np.uint8(1 << (b % 8))
        payload[b // 8] ^= 1 << (b % 8)
        fpay[b // 8] ^= 1 << (b % 8)
    bad = torch.empty(max((ids.size + 31) // 32, 1), dtype=torch.int32, device="cuda")
    nbad = torch.empty(1, dtype=torch.int64, device="cuda")
    plan.unpack_chunks(payload, sums, ids, dst, bad, nbad)
    fbad = plan.empty_bitmap().fill_(-1)
    fnbad = plan.empty_counter().fill_(-1)
    plan.unpack_flagged(fpay, fsums, flagged, dst2, fbad, fnbad, payload_bytes=pb)
    orecv = recv_np.copy()
    obm, onbad = cpu.unpack_chunks(t, C, opay, osums, ids, orecv, oseg)
    torch.cuda.synchronize()
    if recv_np.size:
        assert np.array_equal(to_host(dst)[: recv_np.size], orecv), f"dst {tag}"
        assert np.array_equal(to_host(dst2)[: recv_np.size], orecv), f"flagged dst {tag}"
    want = set(cpu.bitmap_to_set(obm, ids.size))
    assert set(F.bitmap_indices(bad, ids.size).tolist()) == want, tag
    assert int(nbad.item()) == onbad
    # every word of the flagged call's bitmap is written: bits past the list are 0
    assert set(F.bitmap_indices(fbad, plan.n_chunks).tolist()) == want, f"flagged bits {tag}"
    assert int(fnbad.item()) == onbad, tag


def test_delta_bruteforce_tiny_tables():
    rng = np.random.default_rng(71)
    for it in range(400):
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256]))
        nc = cpu.n_chunks(t, C)
        k = int(rng.integers(0, nc + 1))
        ids = np.sort(rng.choice(nc, size=k, replace=False)).astype(np.uint32) if nc else np.zeros(0, np.uint32)
        src = W.random_tiny_state(t, sb, rng)
        recv = rng.integers(0, 256, size=db, dtype=np.uint8)
        _one(t, C, src, recv, ids, rng, f"table {it} C={C} ids={ids.size}")
        if it % 100 == 0:
            log(f"delta tiny {it}")


def test_delta_segment_alignments():
    """Delta lists on plans with explicit segment alignments 16 to 2^20."""
    rng = np.random.default_rng(72)
    for it in range(150):
        seg = int(rng.choice([16, 64, 4096, 1 << 20]))
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256]))
        nc = cpu.n_chunks(t, C)
        k = int(rng.integers(0, nc + 1))
        ids = np.sort(rng.choice(nc, size=k, replace=False)).astype(np.uint32) if nc else np.zeros(0, np.uint32)
        src = W.random_tiny_state(t, sb, rng)
        recv = rng.integers(0, 256, size=db, dtype=np.uint8)
        _one(t, C, src, recv, ids, rng, f"seg {seg} table {it} C={C} ids={ids.size}", seg)
    log("delta segment alignments")


@pytest.mark.parametrize("tile", [0, 2, 4, 5, 9])
def test_delta_every_tile(tile):
    old = os.environ.get("FLASHRESTORE_TILE")
    os.environ["FLASHRESTORE_TILE"] = str(tile)
    try:
        rng = np.random.default_rng(80 + tile)
        for it in range(20):
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=100_000)
            C = int(rng.choice([256, 4096, 16384, 65536]))
            nc = cpu.n_chunks(t, C)
            ids = np.sort(rng.choice(nc, size=int(rng.integers(0, nc + 1)), replace=False)).astype(np.uint32) \
                if nc else np.zeros(0, np.uint32)
            src = W.random_tiny_state(t, sb, rng)
            recv = rng.integers(0, 256, size=db, dtype=np.uint8)
            _one(t, C, src, recv, ids, rng, f"tile {tile} table {it}")
    finally:
        if old is None:
            os.environ.pop("FLASHRESTORE_TILE", None)
        else:
            os.environ["FLASHRESTORE_TILE"] = old


@pytest.mark.parametrize("tile", [0, 1, 2, 3, 5, 8, 9])
def test_delta_capped_grid_multiwave_tiles(tile):
    """Delta calls walk every listed chunk with C / SL workgroup ids, so short
    chunks leave ids that do nothing; under a capped grid one workgroup then
    walks working and idle ids in turn.  With more than one wave per
    workgroup the LDS combine must stay correct across such runs."""
    names = ("FLASHRESTORE_TILE", "FLASHRESTORE_MAX_GRID")
    old = {k: os.environ.get(k) for k in names}
    os.environ["FLASHRESTORE_TILE"] = str(tile)
    try:
        rng = np.random.default_rng(180 + tile)
        for it in range(24):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([1, 2, 3, 7, 64])))
            t, sb, db = W.random_tiny_table(rng, max_entries=10, max_numel=40_000)
            C = int(rng.choice([4096, 16384, 65536]))
            nc = cpu.n_chunks(t, C)
            ids = np.sort(rng.choice(nc, size=int(rng.integers(0, nc + 1)), replace=False)).astype(np.uint32) \
                if nc else np.zeros(0, np.uint32)
            src = W.random_tiny_state(t, sb, rng)
            recv = rng.integers(0, 256, size=db, dtype=np.uint8)
            _one(t, C, src, recv, ids, rng, f"tile {tile} grid {os.environ['FLASHRESTORE_MAX_GRID']} table {it}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def test_flagged_unpack_flags_chunks_past_the_readable_payload():
    """fr_unpack_flagged given fewer payload bytes than the list needs: the
    chunks that lie past them are neither read nor written and are flagged;
    the others are restored and pass."""
    rng = np.random.default_rng(404)
    done = 0
    for it in range(200):
        t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=2000, allow_derive=False)
        C = int(rng.choice([16, 64, 256]))
        _, base, _, _ = cpu.plan(t, C)
        nc = int(base[-1])
        if nc == 0:
            continue
        ids = np.sort(rng.choice(nc, size=int(rng.integers(1, nc + 1)), replace=False)).astype(np.uint32)
        src_np = W.random_tiny_state(t, sb, rng)
        recv_np = rng.integers(0, 256, size=db, dtype=np.uint8)
        off, pb = cpu.delta_layout(t, C, ids)
        opay, osums = cpu.pack_chunks(t, C, src_np, ids)
        limit = int(rng.integers(0, pb + 1))
        plan = F.Plan(t, C, sb, db)
        pay = to_dev(opay[:limit]) if limit else torch.zeros(16, dtype=torch.uint8, device="cuda")
        sums = plan.empty_sums()
        sums[: ids.size] = torch.from_numpy(osums.view(np.int64).reshape(-1, 2)).to("cuda")
        dst = to_dev(recv_np)
        bad, nbad = plan.empty_bitmap(), plan.empty_counter()
        got = plan.unpack_flagged(pay, sums, flagged_bitmap(plan, ids), dst, bad, nbad,
                                  payload_bytes=limit, sync=True)
        exp_dst, exp_bad = recv_np.copy(), set()
        for i, c in enumerate(ids):
            k = int(np.searchsorted(base, c, side="right")) - 1
            e = t[k]
            nb = int(e["numel"]) * (4 if int(e["dtype"]) == W.F32 else 2)
            j = int(c) - int(base[k])
            ln = min(C, nb - j * C)
            if -(-(int(off[i]) + ln) // 16) * 16 <= limit:
                s0, d0 = int(e["src_offset"]) + j * C, int(e["dst_offset"]) + j * C
                exp_dst[d0:d0 + ln] = src_np[s0:s0 + ln]
            else:
                exp_bad.add(i)
        assert set(got.tolist()) == exp_bad and int(nbad.item()) == len(exp_bad), it
        assert np.array_equal(to_host(dst), exp_dst), it
        done += 1
    assert done > 100
    log(f"truncated payloads: {done} lists")


def test_listing_every_chunk_equals_the_full_pack():
    w = W.make_workload(0)
    src = to_dev(W.fill_state(w))
    plan = F.Plan(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
    ids = np.arange(plan.n_chunks, dtype=np.uint32)
    assert plan.delta_layout(ids) == plan.payload_bytes
    p1, s1 = plan.empty_payload().fill_(0xEE), plan.empty_sums()
    p2, s2 = plan.empty_payload().fill_(0x11), plan.empty_sums()
    plan.pack(src, p1, s1)
    plan.pack_chunks(src, ids, p2, s2)
    torch.cuda.synchronize()
    assert torch.equal(p1[: plan.payload_bytes], p2[: plan.payload_bytes]) and torch.equal(s1, s2)


def test_delta_list_errors():
    w = W.make_workload(0)
    plan = F.Plan(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
    for bad in ([3, 3], [5, 4], [plan.n_chunks]):
        with pytest.raises(F.FlashRestoreError) as ei:
            plan.delta_layout(np.array(bad, np.uint32))
        assert ei.value.status == -1


@pytest.mark.timeout(600)
def test_repair_llama8b_share_from_the_flagged_chunks():
    """Donor and a replica with 4096 random flips: compare, re-send only the
    flagged chunks, and the replica equals the donor again."""
    w = W.make_workload(1)
    t, C = w.table, w.chunk_bytes
    donor_np = W.fill_state(w)
    log("generated", w.name)
    plan = F.Plan(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    donor = to_dev(donor_np)
    recv = donor.clone()
    pos = W.flip_positions(donor_np.size * 8, 4096, 4000 + 4096)
    by = (pos // 8).astype(np.int64)
    masks = (np.uint8(1) << (pos % 8).astype(np.uint8)).astype(np.uint8)
    uniq, start = np.unique(by, return_index=True)
    idx = torch.from_numpy(uniq).to("cuda")
    recv[idx] = recv[idx] ^ torch.from_numpy(np.bitwise_or.reduceat(masks, start)).to("cuda")
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    plan.verify_replicas(donor, recv, diff, ndiff)
    ids = F.bitmap_indices(diff, plan.n_chunks).astype(np.uint32)
    assert ids.size == int(ndiff.item()) == 4060
    pb = plan.delta_layout(ids)
    payload = torch.full((pb,), 0xEE, dtype=torch.uint8, device="cuda")
    sums = torch.empty(ids.size, 2, dtype=torch.int64, device="cuda")
    plan.pack_chunks(donor, ids, payload, sums)
    opay, osums = cpu.pack_chunks(t, C, donor_np, ids)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(payload), opay) and np.array_equal(sums_host(sums, ids.size), osums)
    bad = torch.empty((ids.size + 31) // 32, dtype=torch.int32, device="cuda")
    nbad = torch.empty(1, dtype=torch.int64, device="cuda")
    plan.unpack_chunks(payload, sums, ids, recv, bad, nbad)
    plan.verify_replicas(donor, recv, diff, ndiff)
    torch.cuda.synchronize()
    assert int(nbad.item()) == 0 and int(ndiff.item()) == 0 and torch.equal(recv, donor)
    log(f"repaired {ids.size} chunks with {pb} payload bytes")
    # the same repair driven by the compare's device bitmap, no host list
    recv[idx] = recv[idx] ^ torch.from_numpy(np.bitwise_or.reduceat(masks, start)).to("cuda")
    del payload
    fpay = plan.empty_delta_payload()
    fsums = plan.empty_sums()
    counts = torch.empty(2, dtype=torch.int64, device="cuda")
    fbad = plan.empty_bitmap()
    plan.verify_replicas(donor, recv, diff, ndiff)
    plan.pack_flagged(donor, diff, fpay, fsums, counts)
    plan.unpack_flagged(fpay, fsums, diff, recv, fbad, nbad, payload_bytes=fpay.numel())
    torch.cuda.synchronize()
    assert counts.tolist() == [ids.size, pb]
    assert np.array_equal(to_host(fpay[:pb]), opay) and np.array_equal(sums_host(fsums, ids.size), osums)
    assert int(nbad.item()) == 0 and torch.equal(recv, donor)
    log("repaired again from the device bitmap")


@pytest.mark.parametrize("seg", [None, 4096])
@pytest.mark.parametrize("k", [1, 3, 8])
def test_striped_transfer_restores_like_one_payload(k, seg):
    """Multi-donor striping on one GPU: contiguous chunk ranges packed
    separately (C >= the segment alignment) are byte slices of the full
    payload, and placed
    at their offsets they form a buffer that one fr_unpack_state restores to
    the oracle's receiver arena; the gaps between segments are never read."""
    from tests.gpu_util import striped_payload, stripe_ranges

    rng = np.random.default_rng(900 + k)
    cases = []
    for _ in range(4):
        t, sb, db = W.random_tiny_table(rng, max_entries=10, max_numel=60_000)
        cs = [256, 4096, 16384, 65536] if seg is None else [4096, 16384, 65536]
        cases.append((t, int(rng.choice(cs)), W.random_tiny_state(t, sb, rng), sb, db))
    w = W.make_workload(0)
    cases.append((w.table, w.chunk_bytes, W.fill_state(w), w.src_arena_bytes, w.dst_arena_bytes))
    oseg = cpu.SEGMENT if seg is None else seg
    for t, C, src_np, sb, db in cases:
        plan = F.Plan(t, C, sb, db, seg)
        src = to_dev(src_np) if src_np.size else torch.empty(16, dtype=torch.uint8, device="cuda")
        recv, sums, parts = striped_payload(plan, t, src, stripe_ranges(plan.n_chunks, k))
        opay, osums = cpu.pack(t, C, src_np, oseg)
        for (a, b), off, sp, ss in parts:
            assert np.array_equal(sums_host(ss, b - a), osums[2 * a:2 * b])
            if off is not None:
                assert np.array_equal(to_host(sp), opay[off:off + sp.numel()]), (a, b)
        dst = torch.full((max(db, 1),), 0x5A, dtype=torch.uint8, device="cuda")
        bad, nbad = plan.empty_bitmap(), plan.empty_counter()
        plan.unpack(recv, sums, dst, bad, nbad)
        odst = np.full(max(db, 1), 0x5A, np.uint8)
        cpu.unpack(t, C, opay, osums, odst, oseg)
        torch.cuda.synchronize()
        assert int(nbad.item()) == 0 and np.array_equal(to_host(dst), odst)


def test_delta_every_subset_of_a_small_table():
    """All 1,024 lists of a ten-chunk table with a derived parameter, a
    ragged entry, an empty entry and a short bf16 entry, through one plan:
    payload, sums, receiver arena and result set equal the oracle's."""
    from tests.test_oracle_delta import _subset_table

    t, C, sb, db = _subset_table()
    n = cpu.n_chunks(t, C)
    rng = np.random.default_rng(66)
    src_np = W.random_tiny_state(t, sb, rng)
    recv0 = rng.integers(0, 256, size=db, dtype=np.uint8)
    plan = F.Plan(t, C, sb, db)
    src = to_dev(src_np)
    lists = [np.array([c for c in range(n) if mask >> c & 1], dtype=np.uint32) for mask in range(1 << n)]
    # the largest of the lists' payloads
    payload = torch.empty(max(plan.delta_layout(ids) for ids in lists), dtype=torch.uint8, device="cuda")
    sums = torch.empty(n, 2, dtype=torch.int64, device="cuda")
    bad = torch.empty(1, dtype=torch.int32, device="cuda")
    nbad = torch.empty(1, dtype=torch.int64, device="cuda")
    for mask, ids in enumerate(lists):
        pb = plan.delta_layout(ids)
        payload.fill_(0xEE)
        plan.pack_chunks(src, ids, payload, sums)
        opay, osums = cpu.pack_chunks(t, C, src_np, ids)
        assert pb == opay.size
        assert np.array_equal(to_host(payload)[:pb], opay), mask
        assert np.array_equal(sums_host(sums, ids.size), osums), mask
        dst = to_dev(recv0)
        plan.unpack_chunks(payload, sums, ids, dst, bad, nbad)
        orecv = recv0.copy()
        obm, onbad = cpu.unpack_chunks(t, C, opay, osums, ids, orecv)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(dst), orecv), mask
        assert set(F.bitmap_indices(bad, ids.size).tolist()) == set(cpu.bitmap_to_set(obm, ids.size)), mask
        assert int(nbad.item()) == onbad, mask
    log(f"delta subsets {1 << n}")


def test_compare_sums_flags_the_oracle_chunks_and_drives_the_repair():
    """Replicas on different GPUs compare chunk sums, not state:
    fr_compare_sums on the sums of two replicas (each from fr_checksum_state)
    flags the oracle's chunks (replicas that differ in sum alone, in wsum
    alone, in one bit of the last chunk, identical ones, random tables with
    flips), and its bitmap drives fr_pack_flagged / fr_unpack_flagged, which
    restore the replica to the donor.  Raw sums arrays of chunk counts 0 to
    129 (ragged bitmap words) against the oracle's compare."""
    from tests.test_oracle_checksum import _crafted_sums_cases

    t, C, a, cases = _crafted_sums_cases()
    plan = F.Plan(t, C, a.size, a.size)
    sa, sb = plan.empty_sums(), plan.empty_sums()
    bm, nd = plan.empty_bitmap(), plan.empty_counter()
    plan.checksum_state(to_dev(a), sa)
    for name, b, want in cases:
        plan.checksum_state(to_dev(b), sb)
        got = plan.compare_sums(sa, sb, bm, nd, sync=True)
        assert set(got) == want and int(nd.item()) == len(want), name
    rng = np.random.default_rng(1234)
    repaired = 0
    for it in range(30):
        t, nbytes, _ = W.random_tiny_table(rng, max_entries=8, max_numel=3000)
        t["dst_offset"] = t["src_offset"]  # a replica: the donor's layout
        C = int(rng.choice([16, 64, 256, 1024, 4096]))
        x = W.random_tiny_state(t, nbytes, rng)
        inside = np.concatenate([np.arange(int(e["src_offset"]), int(e["src_offset"]) + int(e["numel"]) *
                                           (4 if int(e["dtype"]) == F.FR_F32 else 2)) for e in t] + [np.zeros(0, int)])
        if inside.size == 0:
            continue
        y = x.copy()
        for p in rng.choice(inside, size=int(rng.integers(1, 6))):
            y[p] ^= np.uint8(1 << int(rng.integers(0, 8)))
        plan = F.Plan(t, C, nbytes, nbytes)
        A, B = to_dev(x), to_dev(y)
        sa, sb = plan.empty_sums(), plan.empty_sums()
        bm, nd = plan.empty_bitmap(), plan.empty_counter()
        plan.checksum_state(A, sa)
        plan.checksum_state(B, sb)
        got = plan.compare_sums(sa, sb, bm, nd, sync=True)
        nc = plan.n_chunks
        obm, ond = cpu.compare_sums(cpu.checksum(t, C, x), cpu.checksum(t, C, y))
        assert set(got) == set(cpu.bitmap_to_set(obm, nc)) and int(nd.item()) == ond, (it, C)
        fpay, fsums = plan.empty_delta_payload(), plan.empty_sums()
        counts = torch.empty(2, dtype=torch.int64, device="cuda")
        fbad, fnb = plan.empty_bitmap(), plan.empty_counter()
        plan.pack_flagged(A, bm, fpay, fsums, counts)
        plan.unpack_flagged(fpay, fsums, bm, B, fbad, fnb, payload_bytes=fpay.numel())
        torch.cuda.synchronize()
        assert int(counts[0].item()) == ond and int(fnb.item()) == 0 and torch.equal(B, A), (it, C)
        repaired += 1
    assert repaired > 20
    for n in list(range(0, 70)) + [100, 127, 128, 129]:
        t = np.zeros(1, dtype=W.TABLE_DTYPE)
        t["numel"], t["dtype"], t["derive_from"] = 4 * n, W.F32, -1  # n chunks of 16 bytes
        plan = F.Plan(t, 16, max(16 * n, 16), max(16 * n, 16))
        xs = rng.integers(0, 4, size=2 * n, dtype=np.uint64)
        ys = xs.copy()
        ys[rng.random(2 * n) < 0.15] ^= np.uint64(2)
        X = to_dev(xs.view(np.int64).reshape(-1, 2)) if n else plan.empty_sums()
        Y = to_dev(ys.view(np.int64).reshape(-1, 2)) if n else plan.empty_sums()
        bm, nd = plan.empty_bitmap().fill_(-1), plan.empty_counter().fill_(7)
        got = plan.compare_sums(X, Y, bm, nd, sync=True)
        obm, ond = cpu.compare_sums(xs, ys)
        assert set(got) == set(cpu.bitmap_to_set(obm, n)) and int(nd.item()) == ond, n
        words = to_host(bm).view(np.uint32)[: (n + 31) // 32]
        assert np.array_equal(words, obm), n  # every word written, bits past the last chunk clear
