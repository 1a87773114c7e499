"""Delta repair in the CPU oracle (CPU only): re-sending only the chunks in
which a replica diverged.

Pins: listing every chunk reproduces the full restore's payload and sums
(closed form); a replica repaired from the chunks that the exact compare
flags equals the donor byte for byte; the wire carries exactly the listed
non-derived chunks; a flipped bit on the wire is flagged at its list
position; the C oracle equals the pure-Python oracle on random tables and
lists."""
import numpy as np
import pytest

from oracle import cpu, mini
from paper_2509_03047_amd import workloads as W


def _all_ids(t, C):
    return np.arange(cpu.n_chunks(t, C), dtype=np.uint32)


def test_listing_every_chunk_is_the_full_restore():
    rng = np.random.default_rng(61)
    for _ in range(60):
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256]))
        src = W.random_tiny_state(t, sb, rng)
        fp, fs = cpu.pack(t, C, src)
        dp, ds = cpu.pack_chunks(t, C, src, _all_ids(t, C))
        assert dp.tobytes() == fp.tobytes() and np.array_equal(ds, fs)
    w = W.make_workload(0)
    src = W.fill_state(w)
    fp, fs = cpu.pack(w.table, w.chunk_bytes, src)
    dp, ds = cpu.pack_chunks(w.table, w.chunk_bytes, src, _all_ids(w.table, w.chunk_bytes))
    assert np.array_equal(dp, fp) and np.array_equal(ds, fs)


def _repair(t, C, donor, receiver):
    bm, nd = cpu.verify(t, C, donor, receiver)
    ids = np.array(cpu.bitmap_to_set(bm, cpu.n_chunks(t, C)), dtype=np.uint32)
    pay, sums = cpu.pack_chunks(t, C, donor, ids)
    fixed = receiver.copy()
    rb, nbad = cpu.unpack_chunks(t, C, pay, sums, ids, fixed)
    return ids, pay, fixed, nbad


def test_repair_from_the_flagged_chunks_restores_the_donor():
    w = W.make_workload(0)
    donor = W.fill_state(w)
    t, C = w.table, w.chunk_bytes
    sizes = np.where(t["dtype"] == 1, 4, 2) * t["numel"].astype(np.int64)
    for k in (1, 7, 64, 500):
        recv = donor.copy()
        W.apply_flips(recv, W.flip_positions(donor.size * 8, k, 4000 + k))
        ids, pay, fixed, nbad = _repair(t, C, donor, recv)
        assert nbad == 0 and np.array_equal(fixed, donor)
        # the wire holds exactly the listed chunks of sent (non-derived)
        # entries: a chunk right after the previous sent chunk of its entry
        # follows it, any other starts at a 4 KiB boundary; the end is
        # rounded up to 16
        _, base, _, _ = cpu.plan(t, C)
        end, prev = 0, None
        for c in ids:
            e = int(np.searchsorted(base, int(c), side="right") - 1)
            if int(t[e]["derive_from"]) < 0:
                j = int(c) - int(base[e])
                start = end if prev == (e, j - 1) else -(-end // 4096) * 4096
                end = start + min(C, int(sizes[e]) - j * C)
                prev = (e, j)
        assert pay.size == -(-end // 16) * 16


def test_param_only_divergence_sends_nothing_and_rederives():
    w = W.make_workload(0)
    donor = W.fill_state(w)
    t, C = w.table, w.chunk_bytes
    recv = donor.copy()
    p0 = int(t[0]["src_offset"])  # entry 0 is the embedding's bf16 param
    recv[p0 + 5] ^= 0x10
    recv[p0 + 70000] ^= 0x01
    ids, pay, fixed, nbad = _repair(t, C, donor, recv)
    assert list(ids) == [0, 1] and pay.size == 0
    assert nbad == 0 and np.array_equal(fixed, donor)


def test_master_divergence_repairs_master_and_param():
    w = W.make_workload(0)
    donor = W.fill_state(w)
    t, C = w.table, w.chunk_bytes
    recv = donor.copy()
    m0, p0 = int(t[1]["src_offset"]), int(t[0]["src_offset"])
    recv[m0 + 3] ^= 0x40  # exponent bit of master element 0
    recv[p0 + 1] ^= 0x40  # and its bf16 image
    ids, pay, fixed, nbad = _repair(t, C, donor, recv)
    assert nbad == 0 and np.array_equal(fixed, donor)


def test_wire_flip_is_flagged_at_its_list_position():
    w = W.make_workload(0)
    donor = W.fill_state(w)
    t, C = w.table, w.chunk_bytes
    ids = np.array([2, 3, 10, 11, 40, 400, 803], dtype=np.uint32)
    pay, sums = cpu.pack_chunks(t, C, donor, ids)
    off, pb = cpu.delta_layout(t, C, ids)
    _, base, _, _ = cpu.plan(t, C)
    sizes = np.where(t["dtype"] == 1, 4, 2) * t["numel"].astype(np.int64)
    lens = []
    for c in ids:
        e = int(np.searchsorted(base, int(c), side="right") - 1)
        lens.append(min(C, int(sizes[e]) - (int(c) - int(base[e])) * C))
    sent = [i for i in range(ids.size) if off[i] != cpu.NO_PAYLOAD]
    assert sent  # the list mixes derived (not sent) and sent chunks
    assert len(sent) < ids.size
    rng = np.random.default_rng(62)
    for _ in range(40):
        b = int(rng.integers(0, pb * 8))
        p = pay.copy()
        p[b // 8] ^= np.uint8(1 << (b % 8))
        recv = donor.copy()
        bm, nbad = cpu.unpack_chunks(t, C, p, sums, ids, recv)
        exp = {i for i in sent if off[i] <= b // 8 < off[i] + lens[i]}  # padding bytes are not data
        assert set(cpu.bitmap_to_set(bm, ids.size)) == exp and nbad == len(exp)


def test_bad_lists_are_rejected():
    t, sb, db = W.random_tiny_table(np.random.default_rng(63), max_entries=3, max_numel=200)
    n = cpu.n_chunks(t, 16)
    for bad in ([1, 1], [2, 1], [n]):
        try:
            cpu.delta_layout(t, 16, np.array(bad, np.uint32))
            raise AssertionError("accepted", bad)
        except ValueError:
            pass


def test_c_oracle_equals_python_oracle_on_delta():
    rng = np.random.default_rng(64)
    for _ in range(400):
        t, sb, db = W.random_tiny_table(rng, max_numel=150)
        C = int(rng.choice([16, 32, 64, 256]))
        nc = cpu.n_chunks(t, C)
        if nc == 0:
            continue
        ids = np.sort(rng.choice(nc, size=int(rng.integers(1, nc + 1)), replace=False)).astype(np.uint32)
        src = W.random_tiny_state(t, sb, rng)
        pay, sums = cpu.pack_chunks(t, C, src, ids)
        mp, ms = mini.pack_chunks(t, C, src.tobytes(), [int(i) for i in ids])
        assert pay.tobytes() == mp
        assert [tuple(int(x) for x in sums[2 * i:2 * i + 2]) for i in range(ids.size)] == ms
        recv = rng.integers(0, 256, size=db, dtype=np.uint8)
        mrecv = bytearray(recv.tobytes())
        p = pay.copy()
        if p.size and rng.random() < 0.5:
            b = int(rng.integers(0, p.size * 8))
            p[b // 8] ^= np.uint8(1 << (b % 8))
        bm, nbad = cpu.unpack_chunks(t, C, p, sums, ids, recv)
        mbad = mini.unpack_chunks(t, C, p.tobytes(), ms, [int(i) for i in ids], mrecv)
        assert recv.tobytes() == bytes(mrecv)
        assert set(cpu.bitmap_to_set(bm, ids.size)) == mbad and nbad == len(mbad)


def _stripe_cuts(n, k, rng):
    """k contiguous chunk ranges covering [0, n) (some may be empty)."""
    cuts = np.sort(rng.integers(0, n + 1, size=k - 1)) if n else np.zeros(k - 1, np.int64)
    edges = [0] + [int(c) for c in cuts] + [n]
    return list(zip(edges[:-1], edges[1:]))


def _chunk_payload_offset(t, C, c, seg=cpu.SEGMENT):
    """Full-payload offset of global chunk c (None for a derived chunk)."""
    _, base, pay, _ = cpu.plan(t, C, seg)
    k = int(np.searchsorted(base, c, side="right") - 1)
    if int(t[k]["derive_from"]) >= 0:
        return None
    return int(pay[k]) + (c - int(base[k])) * C


@pytest.mark.parametrize("seg", [16, 4096])
def test_stripes_are_slices_of_the_full_payload(seg):
    """With C >= the segment alignment every chunk starts on a segment
    boundary of the full payload, so the delta payload of a contiguous chunk
    range (a stripe)
    is the full payload's bytes from the range's first sent chunk on, and
    its sums are the full sums of the range: stripes packed separately (one
    per donor) and placed at those offsets form a buffer that a whole
    unpack restores exactly (it never reads the gaps between segments)."""
    rng = np.random.default_rng(313)
    cases = []
    for _ in range(20):
        t, sb, db = W.random_tiny_table(rng, max_entries=10, max_numel=60_000)
        cs = [16, 256, 4096, 65536] if seg == 16 else [4096, 16384, 65536]
        cases.append((t, int(rng.choice(cs)), W.random_tiny_state(t, sb, rng), db))
    w = W.make_workload(0)
    cases.append((w.table, w.chunk_bytes, W.fill_state(w), w.dst_arena_bytes))
    for t, C, src, db in cases:
        fp, fs = cpu.pack(t, C, src, seg)
        n = cpu.n_chunks(t, C)
        buf = np.full(fp.size, 0xEE, np.uint8)  # gap bytes never written
        got_sums = np.zeros_like(fs)
        for a, b in _stripe_cuts(n, int(rng.integers(1, 9)), rng):
            ids = np.arange(a, b, dtype=np.uint32)
            dp, ds = cpu.pack_chunks(t, C, src, ids, seg)
            assert np.array_equal(ds, fs[2 * a:2 * b])
            got_sums[2 * a:2 * b] = ds
            offs = [o for o in (_chunk_payload_offset(t, C, int(c), seg) for c in ids) if o is not None]
            if not offs:  # only derived chunks: nothing on the wire
                assert dp.size == 0
                continue
            assert np.array_equal(dp, fp[offs[0]:offs[0] + dp.size]), (a, b)
            buf[offs[0]:offs[0] + dp.size] = dp
        ref = np.zeros(max(db, 1), np.uint8)
        cpu.unpack(t, C, fp, fs, ref, seg)
        dst = np.zeros(max(db, 1), np.uint8)
        bm, nbad = cpu.unpack(t, C, buf, got_sums, dst, seg)
        assert nbad == 0 and np.array_equal(dst, ref)


def test_stripes_below_the_segment_alignment_are_not_slices():
    """The slice property needs C >= the segment alignment: with 1 KiB chunks
    and 4 KiB segments a stripe starting inside an entry is not 4 KiB-aligned
    in the full payload, so the next entry's segment lands elsewhere (the
    reading is checked, not assumed); with 16-byte segments it holds."""
    t = np.array([(0, 0, 3000, W.F32, -1), (12288, 12288, 3000, W.F32, -1)], dtype=W.TABLE_DTYPE)
    C = 1024
    src = np.arange(24576, dtype=np.uint32).astype(np.uint8)
    ids = np.arange(1, cpu.n_chunks(t, C), dtype=np.uint32)  # from chunk 1 of entry 0
    fp, _ = cpu.pack(t, C, src, 4096)
    dp, _ = cpu.pack_chunks(t, C, src, ids, 4096)
    off = _chunk_payload_offset(t, C, 1, 4096)
    assert off == 1024 and not np.array_equal(dp, fp[off:off + dp.size])
    fp, _ = cpu.pack(t, C, src)
    dp, _ = cpu.pack_chunks(t, C, src, ids)
    off = _chunk_payload_offset(t, C, 1)
    assert off == 1024 and np.array_equal(dp, fp[off:off + dp.size])


def _subset_table():
    """Ten chunks of 64 bytes: a bf16 parameter (2 chunks) derived from its
    master (4 chunks), a plain fp32 entry of 2 chunks and 1 ragged one, an
    empty entry, and a bf16 entry of one short chunk."""
    t = np.array([(0, 0, 60, W.BF16, 1), (128, 128, 60, W.F32, -1), (384, 400, 40, W.F32, -1),
                  (544, 560, 0, W.F32, -1), (544, 576, 5, W.BF16, -1)], dtype=W.TABLE_DTYPE)
    return t, 64, 560, 608


def test_every_delta_subset_of_a_small_table():
    """All 1,024 lists of the ten chunks: the C oracle's delta layout,
    payload, sums and repair equal the pure-Python oracle's."""
    t, C, sb, db = _subset_table()
    n = cpu.n_chunks(t, C)
    assert n == 10
    rng = np.random.default_rng(65)
    src = W.random_tiny_state(t, sb, rng)
    recv0 = rng.integers(0, 256, size=db, dtype=np.uint8)
    for mask in range(1 << n):
        ids = np.array([c for c in range(n) if mask >> c & 1], dtype=np.uint32)
        off, pb = cpu.delta_layout(t, C, ids)
        moff, mpb = mini._delta_offsets(t, C, [int(i) for i in ids])
        assert pb == mpb and [None if o == cpu.NO_PAYLOAD else int(o) for o in off] == moff, mask
        pay, sums = cpu.pack_chunks(t, C, src, ids)
        mp, ms = mini.pack_chunks(t, C, src.tobytes(), [int(i) for i in ids])
        assert pay.tobytes() == mp and [tuple(int(x) for x in sums[2 * i:2 * i + 2]) for i in range(ids.size)] == ms
        recv, mrecv = recv0.copy(), bytearray(recv0.tobytes())
        bm, nbad = cpu.unpack_chunks(t, C, pay, sums, ids, recv)
        mbad = mini.unpack_chunks(t, C, pay.tobytes(), ms, [int(i) for i in ids], mrecv)
        assert recv.tobytes() == bytes(mrecv) and set(cpu.bitmap_to_set(bm, ids.size)) == mbad, mask
