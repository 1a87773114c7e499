"""GPU parity on small inputs: the HIP path through the C ABI vs the CPU
oracle, bit for bit (payload, sums, receiver arena with canaries, bitmaps,
counts), plus fault injection, determinism and error behaviour."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests.gpu_util import Restore, log, sums_host, to_dev, to_host  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_03047_amd import flashrestore  # noqa: F401  (fails loudly if unbuilt)


def _check_against_oracle(t, C, src_np, src_bytes, dst_bytes, corrupt_rng=None, tag="", seg=None):
    """seg: payload segment alignment (None: the default, 16)."""
    r = Restore(t, C, src_bytes, dst_bytes, seg=seg)
    oseg = cpu.SEGMENT if seg is None else seg
    src = to_dev(src_np) if src_np.size else torch.empty(1, dtype=torch.uint8, device="cuda")
    r.pack(src)
    pay, sums = cpu.pack(t, C, src_np, oseg)
    nc = r.n_chunks
    g_pay = to_host(r.payload)[: pay.size]
    g_sums = sums_host(r.sums, nc)
    assert np.array_equal(g_pay, pay), f"payload {tag}"
    assert np.array_equal(g_sums, sums), f"sums {tag}"
    # optionally corrupt the wire
    if corrupt_rng is not None and pay.size and corrupt_rng.random() < 0.5:
        b = int(corrupt_rng.integers(0, pay.size * 8))
        pay[b // 8] ^= np.uint8(1 << (b % 8))
        r.payload[b // 8] ^= 1 << (b % 8)
    if corrupt_rng is not None and nc and corrupt_rng.random() < 0.25:
        c = int(corrupt_rng.integers(0, nc))
        sums[2 * c] ^= np.uint64(1)
        r.sums[c, 0] ^= 1
    r.unpack()
    dst = np.full(max(dst_bytes, 1), 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst, oseg)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(r.dst), dst), f"dst {tag}"
    assert r.bad_set() == set(cpu.bitmap_to_set(bm, nc)), f"bad set {tag}"
    assert int(r.n_bad.item()) == nbad
    # verify the restored replica against the sender (same layout only) and a flipped copy
    b_np = src_np.copy()
    if b_np.size:
        for _ in range(int((corrupt_rng or np.random.default_rng(0)).integers(0, 3))):
            b = int((corrupt_rng or np.random.default_rng(0)).integers(0, b_np.size * 8))
            b_np[b // 8] ^= np.uint8(1 << (b % 8))
    bd = to_dev(b_np) if b_np.size else torch.empty(1, dtype=torch.uint8, device="cuda")
    sa, sb = r.plan.empty_sums(), r.plan.empty_sums()
    r.verify(src, bd, sa, sb)
    vbm, nd, osa, osb = cpu.verify(t, C, src_np, b_np, with_sums=True)
    assert r.diff_set() == set(cpu.bitmap_to_set(vbm, nc)), f"diff {tag}"
    assert int(r.n_diff.item()) == nd
    assert np.array_equal(sums_host(sa, nc), osa) and np.array_equal(sums_host(sb, nc), osb)
    r.verify(src, bd)  # without sums: same set
    assert r.diff_set() == set(cpu.bitmap_to_set(vbm, nc))
    r.checksum(src)
    torch.cuda.synchronize()
    assert np.array_equal(sums_host(r.csum, nc), cpu.checksum(t, C, src_np))


def test_bruteforce_tiny_tables():
    rng = np.random.default_rng(1234)
    n = 1000
    for it in range(n):
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256]))
        src = W.random_tiny_state(t, sb, rng)
        _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"table {it} C={C}")
        if it % 200 == 0:
            log(f"tiny table {it}/{n}")


def test_bruteforce_multi_tile_ragged():
    """Tables whose chunks span several workgroup passes with ragged tails."""
    rng = np.random.default_rng(99)
    for it in range(40):
        t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=300_000)
        C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
        src = W.random_tiny_state(t, sb, rng)
        _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"multi {it} C={C}")


@pytest.mark.parametrize("seg", [16, 32, 256, 4096, 1 << 20])
def test_segment_alignments_match_oracle(seg):
    """Plans with an explicit payload segment alignment (fr_plan_create_ex):
    tiny tables and multi-slice tables with ragged tails, bit for bit
    against the oracle at the same alignment."""
    rng = np.random.default_rng(500 + seg.bit_length())
    for it in range(120):
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256]))
        src = W.random_tiny_state(t, sb, rng)
        _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"seg {seg} table {it} C={C}", seg=seg)
    for it in range(8):
        t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=300_000)
        C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
        src = W.random_tiny_state(t, sb, rng)
        _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"seg {seg} multi {it} C={C}", seg=seg)
    log(f"segment alignment {seg}")


def test_toy_decoder_full_parity():
    w = W.make_workload(0)
    src = W.fill_state(w)
    log("toy decoder", w.n_params, "params")
    _check_against_oracle(w.table, w.chunk_bytes, src, w.src_arena_bytes, w.dst_arena_bytes, tag="toy")
    # exact round trip and nothing flagged
    r = Restore(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
    s = to_dev(src)
    r.pack(s)
    r.unpack()
    torch.cuda.synchronize()
    assert torch.equal(r.dst, s) and int(r.n_bad.item()) == 0


def test_fault_injection_toy_exact_sets():
    """Single flips in the payload, the sums, the sender's param or master:
    the GPU flags exactly the oracle's chunks."""
    w = W.make_workload(0)
    src = W.fill_state(w)
    t, C = w.table, w.chunk_bytes
    rng = np.random.default_rng(7)
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    s = to_dev(src)
    r.pack(s)
    pay, sums = cpu.pack(t, C, src)
    nc = r.n_chunks
    for _ in range(24):  # payload flips
        b = int(rng.integers(0, pay.size * 8))
        p = pay.copy()
        p[b // 8] ^= np.uint8(1 << (b % 8))
        gp = r.payload.clone()
        gp[b // 8] ^= 1 << (b % 8)
        r.unpack(payload=gp)
        bm, nbad = cpu.unpack(t, C, p, sums, np.zeros(w.dst_arena_bytes, np.uint8))
        assert r.bad_set() == set(cpu.bitmap_to_set(bm, nc)) and nbad >= 1
    for _ in range(8):  # sums flips
        c = int(rng.integers(0, nc))
        gs = r.sums.clone()
        gs[c, int(rng.integers(0, 2))] ^= 1 << int(rng.integers(0, 63))
        r.unpack(sums=gs)
        assert r.bad_set() == {c}
    for _ in range(24):  # sender-side flips before pack (any of the 4 arrays)
        b = int(rng.integers(0, src.size * 8))
        s2 = src.copy()
        s2[b // 8] ^= np.uint8(1 << (b % 8))
        p, sm = cpu.pack(t, C, s2)
        bm, _ = cpu.unpack(t, C, p, sm, np.zeros(w.dst_arena_bytes, np.uint8))
        g2 = s.clone()
        g2[b // 8] ^= 1 << (b % 8)
        r.pack(g2)
        r.unpack()
        assert r.bad_set() == set(cpu.bitmap_to_set(bm, nc))


def test_deterministic_across_grid_sizes():
    w = W.make_workload(0)
    src = to_dev(W.fill_state(w))
    outs = []
    old = os.environ.get("FLASHRESTORE_MAX_GRID")
    try:
        for g in ("1", "7", "300", ""):
            os.environ["FLASHRESTORE_MAX_GRID"] = g
            r = Restore(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
            gp = None
            r.pack(src)
            gp = r.payload.clone()
            gp[12345] ^= 4  # one bad chunk
            r.unpack(payload=gp)
            r.verify(src, r.dst)
            torch.cuda.synchronize()
            outs.append((r.payload.cpu(), r.sums.cpu(), r.dst.cpu(), r.bad.cpu(), r.n_bad.cpu(), r.diff.cpu()))
    finally:
        if old is None:
            os.environ.pop("FLASHRESTORE_MAX_GRID", None)
        else:
            os.environ["FLASHRESTORE_MAX_GRID"] = old
    for o in outs[1:]:
        for x, y in zip(outs[0], o):
            assert torch.equal(x, y)
    assert int(outs[0][4].item()) >= 1


def test_empty_and_zero_length_tables():
    from paper_2509_03047_amd import flashrestore as F

    for rows in ([], [(0, 0, 0, 1, -1), (16, 16, 0, 2, -1)]):
        t = F.as_table(rows) if rows else np.zeros(0, dtype=F.DESC_DTYPE)
        r = Restore(t, 64, 64, 64)
        assert r.n_chunks == 0 and r.plan.payload_bytes == 0
        src = torch.zeros(64, dtype=torch.uint8, device="cuda")
        r.n_bad.fill_(77)
        r.pack(src)
        r.unpack()
        r.verify(src, src)
        r.checksum(src)
        torch.cuda.synchronize()
        assert int(r.n_bad.item()) == 0 and int(r.n_diff.item()) == 0
        assert torch.all(r.dst == 0xA5)


@pytest.mark.parametrize("tile", list(range(11)))
def test_every_tile_matches_oracle(tile):
    """Each launch tile (threads x vectors per slice) gives the oracle's bytes."""
    old = os.environ.get("FLASHRESTORE_TILE")
    os.environ["FLASHRESTORE_TILE"] = str(tile)
    try:
        rng = np.random.default_rng(500 + tile)
        for it in range(60):
            t, sb, db = W.random_tiny_table(rng)
            C = int(rng.choice([16, 64, 256, 1024, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"tile {tile} table {it} C={C}")
        for it in range(5):
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=200_000)
            C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"tile {tile} multi {it} C={C}")
    finally:
        if old is None:
            os.environ.pop("FLASHRESTORE_TILE", None)
        else:
            os.environ["FLASHRESTORE_TILE"] = old


def _short_chunk_table(rng, scale=1):
    """Entries (bf16 parameter derived from its master, two plain fp32) whose
    last chunk of C = 16 KiB * scale holds every number of 4 KiB * scale
    slices, with ragged tails; the receiver gaps differ from the sender's."""
    from paper_2509_03047_amd import flashrestore as F

    numels = [1, 3, 511, 512, 513, 1023, 1024, 1025, 2047, 2048, 3071, 4095, 4096, 4097,
              6143, 8191, 8193, 12289, 16383]
    numels = [n * scale + (scale - 1) * (k % 3) for k, n in enumerate(numels)]
    rows, so, do = [], 0, 0
    for n in numels:
        for dtype, derive in ((F.FR_BF16, len(rows) + 1), (F.FR_F32, -1), (F.FR_F32, -1)):
            nb = n * (4 if dtype == F.FR_F32 else 2)
            gap = 16 * int(rng.integers(0, 5))
            rows.append((so, do + gap, n, dtype, derive))
            so += (nb + 15) // 16 * 16
            do += gap + (nb + 15) // 16 * 16
    t = F.as_table(rows)
    src = np.zeros(so, np.uint8)
    for k, (s_off, _, n, dtype, derive) in enumerate(rows):
        if dtype == F.FR_F32:
            src[s_off:s_off + 4 * n] = rng.standard_normal(n).astype(np.float32).view(np.uint8)
    for k, (s_off, _, n, dtype, derive) in enumerate(rows):
        if derive >= 0:
            m_off = rows[derive][0]
            master = src[m_off:m_off + 4 * n].view(np.float32)
            src[s_off:s_off + 2 * n] = W._bf16_round(master).view(np.uint8)
    return t, src, so, do


def test_short_last_chunks_every_slot_count():
    """Entries whose last chunk holds every possible number of 4 KiB slices
    (and ragged tails inside them), for plain chunks and for bf16 parameter
    chunks derived from masters, with the receiver laid out differently from
    the sender: the walk lists only the slices a short chunk has."""
    rng = np.random.default_rng(77)
    t, src, so, do = _short_chunk_table(rng)
    C = 1 << 14  # four slices per chunk at the default tiles
    _check_against_oracle(t, C, src, so, do, corrupt_rng=rng, tag="short chunks")


def _slice_count_table(rng, C, SL):
    """Triples (bf16 parameter derived from its master, the master, a plain
    fp32 entry) of one whole chunk plus a short chunk of every slice count
    1 .. C / SL, ending on a slice boundary or ragged inside its last slice
    (12 bytes short, half a slice past); the derived group then walks every
    count SPC + k.  The receiver gaps differ from the sender's."""
    from paper_2509_03047_amd import flashrestore as F

    rows, so, do = [], 0, 0
    for k in range(1, C // SL + 1):
        for short in sorted({0, 12, SL // 2 - 4}):
            n = (C + k * SL - short) // 4
            for dtype, derive in ((F.FR_BF16, len(rows) + 1), (F.FR_F32, -1), (F.FR_F32, -1)):
                nb = n * (4 if dtype == F.FR_F32 else 2)
                gap = 16 * int(rng.integers(0, 5))
                rows.append((so, do + gap, n, dtype, derive))
                so += (nb + 15) // 16 * 16
                do += gap + (nb + 15) // 16 * 16
    t = F.as_table(rows)
    src = np.zeros(so, np.uint8)
    for s_off, _, n, dtype, derive in rows:
        if dtype == F.FR_F32:
            src[s_off:s_off + 4 * n] = rng.standard_normal(n).astype(np.float32).view(np.uint8)
    for s_off, _, n, dtype, derive in rows:
        if derive >= 0:
            m_off = rows[derive][0]
            src[s_off:s_off + 2 * n] = W._bf16_round(src[m_off:m_off + 4 * n].view(np.float32)).view(np.uint8)
    return t, src, so, do


# slice bytes of the tiles: 3: 16 KiB, 4: 4 KiB, 5: 4 KiB, 7: 1 KiB, 10: 8 KiB
SLICE_BYTES = {3: 16384, 4: 4096, 5: 4096, 7: 1024, 10: 8192}


@pytest.mark.parametrize("tile", sorted(SLICE_BYTES))
def test_every_slice_count_per_tile(tile):
    """For each tile: a table whose short chunks hold every slice count (plain
    and derived), random tables with C up to 1 MiB, and delta lists (implicit
    walks) give the oracle's bytes."""
    old = os.environ.get("FLASHRESTORE_TILE")
    os.environ["FLASHRESTORE_TILE"] = str(tile)
    rng = np.random.default_rng(600 + tile)
    try:
        C = 1 << 16
        t, src, so, do = _slice_count_table(rng, C, SLICE_BYTES[tile])
        _check_against_oracle(t, C, src, so, do, corrupt_rng=rng, tag=f"tile {tile} slice counts")
        _delta_against_oracle(t, C, src, so, do, rng, f"tile {tile} slice counts")
        for it in range(4):
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=200_000)
            C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"tile {tile} multi {it}")
            _delta_against_oracle(t, C, src, sb, db, rng, f"tile {tile} multi {it}")
    finally:
        if old is None:
            os.environ.pop("FLASHRESTORE_TILE", None)
        else:
            os.environ["FLASHRESTORE_TILE"] = old


@pytest.mark.parametrize("tile", [0, 3, 4, 5, 7, 10])
@pytest.mark.parametrize("absorb", ["0", "1"])
@pytest.mark.parametrize("line", ["1", "2", "3"])
def test_line_aligned_walks_match_oracle(tile, line, absorb):
    """Line-aligned walks (every slice cut at a 128-byte line, one more
    slice for a chunk that starts inside a line) give the oracle's bytes:
    line 1 cuts pack, compare and checksum at lines of the arena read and
    unpack's plain chunks at lines of the receiver, line 2 cuts pack and
    unpack at lines of the payload (the compare and checksum at arena
    lines), line 3 cuts pack and unpack's plain chunks at slice boundaries
    of the payload (one more slice for a chunk that starts inside a slice;
    the compare and checksum at arena lines); with absorb, every operation's
    chunks keep their plain slice count and the last slice takes the
    leftover lead.  Random tables at random 16-byte offsets
    (16-byte payload
    segments, so payload chunks start inside lines too), chunks from 16 B
    (several chunks per line) to 1 MiB, and short chunks of every slice
    count."""
    absorbs = tuple(f"FLASHRESTORE_ABSORB_{op}" for op in ("PACK", "UNPACK", "VERIFY", "CHECKSUM"))
    names = ("FLASHRESTORE_TILE", "FLASHRESTORE_LINE", "FLASHRESTORE_MAX_GRID") + absorbs
    old = {k: os.environ.get(k) for k in names}
    os.environ["FLASHRESTORE_TILE"], os.environ["FLASHRESTORE_LINE"] = str(tile), line
    for k in absorbs:
        os.environ[k] = absorb
    rng = np.random.default_rng(700 + tile + 50 * int(line) + 1000 * int(absorb))
    try:
        for it in range(40):
            # grid-stride launches too (a capped grid walks several slices per workgroup)
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 1, 7, 300])))
            t, sb, db = W.random_tiny_table(rng)
            C = int(rng.choice([16, 32, 64, 256, 1024]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"line tile {tile} table {it} C={C}")
        for it in range(6):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 7, 300])))
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=200_000)
            C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"line tile {tile} multi {it} C={C}")
            _delta_against_oracle(t, C, src, sb, db, rng, f"line tile {tile} multi {it}")
        if tile in SLICE_BYTES:
            os.environ["FLASHRESTORE_MAX_GRID"] = "0"
            t, src, so, do = _slice_count_table(rng, 1 << 16, SLICE_BYTES[tile])
            _check_against_oracle(t, 1 << 16, src, so, do, corrupt_rng=rng, tag=f"line tile {tile} slice counts")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("tile", [0, 3, 4, 5, 7, 10])
def test_payload_block_walks_match_oracle(tile):
    """Pack and unpack walked by blocks of the payload (each workgroup moves
    one whole tile of the payload, across chunk and entry boundaries), forced
    whatever the table's alignment, give the oracle's payload, sums, receiver
    arena and bad sets: random tables at random 16-byte offsets with derived
    entries (pack sums them, and unpack restores them with their masters, in
    slice walks of their own), chunks from 16 B (many chunks per block) to
    1 MiB, segment alignments 16, 64 and 4096 (zero gaps inside blocks),
    capped grids, short chunks of every slice count, corrupted wires, and
    tables with nothing to send."""
    names = ("FLASHRESTORE_TILE", "FLASHRESTORE_LINE_PACK", "FLASHRESTORE_LINE_UNPACK",
             "FLASHRESTORE_MAX_GRID")
    old = {k: os.environ.get(k) for k in names}
    os.environ["FLASHRESTORE_TILE"] = str(tile)
    os.environ["FLASHRESTORE_LINE_PACK"] = os.environ["FLASHRESTORE_LINE_UNPACK"] = "4"
    rng = np.random.default_rng(900 + tile)
    try:
        for it in range(40):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 1, 7, 300])))
            t, sb, db = W.random_tiny_table(rng)
            C = int(rng.choice([16, 32, 64, 256, 1024]))
            seg = int(rng.choice([16, 16, 64, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, seg=seg,
                                  tag=f"blocks tile {tile} table {it} C={C} seg={seg}")
        for it in range(6):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 7, 300])))
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=200_000)
            C = int(rng.choice([4096, 16384, 65536, 1 << 20]))
            seg = int(rng.choice([16, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, seg=seg,
                                  tag=f"blocks tile {tile} multi {it} C={C} seg={seg}")
        if tile in SLICE_BYTES:
            os.environ["FLASHRESTORE_MAX_GRID"] = "0"
            t, src, so, do = _slice_count_table(rng, 1 << 16, SLICE_BYTES[tile])
            _check_against_oracle(t, 1 << 16, src, so, do, corrupt_rng=rng, tag=f"blocks tile {tile} slice counts")
        # no derived entries (no slice walk in the launch), and only empty entries
        for max_numel in (300, 0):
            t, sb, db = W.random_tiny_table(rng, max_numel=max_numel, allow_derive=False)
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, 64, src, sb, db, corrupt_rng=rng, tag=f"blocks tile {tile} plain {max_numel}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _overlapping_sender_table(rng, n_max=10, max_numel=3000):
    """Entries whose sender ranges overlap (the sender arena is about half
    the bytes the entries read; any 16-byte offset), receiver ranges apart.
    No derived entries."""
    n = int(rng.integers(2, n_max + 1))
    numel = rng.integers(0, max_numel + 1, size=n).astype(np.uint64)
    dts = np.where(rng.random(n) < 0.5, W.F32, W.BF16).astype(np.uint32)
    nbytes = numel * np.where(dts == W.F32, 4, 2).astype(np.uint64)
    span = max(16, int(nbytes.sum()) // 32 * 16)
    src_off = np.array([int(rng.integers(0, span // 16 + 1)) * 16 for _ in range(n)], dtype=np.uint64)
    sb = int(max(int(src_off[k] + nbytes[k]) for k in range(n)))
    sb = -(-sb // 16) * 16
    dst_off, db = W._scatter_layout(nbytes, rng)
    t = np.zeros(n, dtype=W.TABLE_DTYPE)
    t["src_offset"], t["dst_offset"], t["numel"], t["dtype"] = src_off, dst_off, numel, dts
    t["derive_from"] = -1
    return t, sb, int(db)


WALK_SETS = {
    "default": {},
    "lines": {"FLASHRESTORE_LINE": "1"},
    "payload tiles": {"FLASHRESTORE_LINE_PACK": "4", "FLASHRESTORE_LINE_UNPACK": "4"},
    "slices": {"FLASHRESTORE_LINE": "0"},
    "buffer loads": {"FLASHRESTORE_BUF_PACK": "1", "FLASHRESTORE_BUF_UNPACK": "1",
                     "FLASHRESTORE_BUF_VERIFY": "1", "FLASHRESTORE_BUF_CHECKSUM": "1"},
}


@pytest.mark.parametrize("walks", sorted(WALK_SETS))
@pytest.mark.parametrize("tile", [None, 3, 7])
def test_overlapping_sender_ranges_match_oracle(walks, tile):
    """Entries may read the same sender bytes (their receiver ranges stay
    apart): pack, unpack, compare and checksum give the oracle's payload,
    sums, receiver arena and bad sets when sender ranges overlap, at any
    16-byte offset, from tiny chunks (many per slice) to large ones, with
    capped grids, under every walk."""
    names = ("FLASHRESTORE_TILE", "FLASHRESTORE_MAX_GRID") + tuple(
        {k for env in WALK_SETS.values() for k in env})
    old = {k: os.environ.get(k) for k in names}
    for k in names:
        os.environ.pop(k, None)
    os.environ.update(WALK_SETS[walks])
    if tile is not None:
        os.environ["FLASHRESTORE_TILE"] = str(tile)
    rng = np.random.default_rng(1700 + (tile or 0) + 31 * sorted(WALK_SETS).index(walks))
    try:
        for it in range(10):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 0, 7])))
            t, sb, db = _overlapping_sender_table(rng, max_numel=int(rng.choice([300, 30_000])))
            C = int(rng.choice([16, 64, 1024, 16384]))
            src = rng.integers(0, 256, size=sb, dtype=np.uint8)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng,
                                  tag=f"overlap {walks} tile {tile} table {it} C={C}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("tile", [3, 4, 5, 7])
@pytest.mark.parametrize("line", ["0", "1", "2"])
def test_buffer_load_slices_match_oracle(tile, line):
    """The slice kernels loading through buffer resources (the option that
    keeps every load of a thread in flight: lanes outside a chunk's data load
    zeros) give the oracle's bytes for all four operations and the delta
    calls, on slice walks plain and cut at lines (tile walks off)."""
    ops = ("PACK", "UNPACK", "VERIFY", "CHECKSUM")
    names = ("FLASHRESTORE_TILE", "FLASHRESTORE_LINE", "FLASHRESTORE_ABSORB_PACK",
             "FLASHRESTORE_ABSORB_UNPACK") + tuple(f"FLASHRESTORE_BUF_{op}" for op in ops)
    old = {k: os.environ.get(k) for k in names}
    os.environ["FLASHRESTORE_TILE"], os.environ["FLASHRESTORE_LINE"] = str(tile), line
    for op in ops:
        os.environ[f"FLASHRESTORE_BUF_{op}"] = "1"
    rng = np.random.default_rng(1300 + tile + 10 * int(line))
    try:
        for it in range(16):
            os.environ["FLASHRESTORE_ABSORB_PACK"] = os.environ["FLASHRESTORE_ABSORB_UNPACK"] = str(it % 2)
            t, sb, db = W.random_tiny_table(rng)
            C = int(rng.choice([16, 64, 256, 1024]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"buf tile {tile} line {line} {it}")
        for it in range(3):
            t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=200_000)
            C = int(rng.choice([4096, 65536, 1 << 20]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"buf tile {tile} multi {it}")
            _delta_against_oracle(t, C, src, sb, db, rng, f"buf tile {tile} multi {it}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("order", ["0", "1"])
def test_walk_orders_match_oracle(order):
    """The compare and the checksum walking the arena in chunk order or in
    arena address order (tables list their tensors in shuffled arena order)
    give the oracle's sets and sums, also under capped grids."""
    names = ("FLASHRESTORE_ORDER_VERIFY", "FLASHRESTORE_ORDER_CHECKSUM", "FLASHRESTORE_MAX_GRID")
    old = {k: os.environ.get(k) for k in names}
    os.environ["FLASHRESTORE_ORDER_VERIFY"] = os.environ["FLASHRESTORE_ORDER_CHECKSUM"] = order
    rng = np.random.default_rng(1400 + int(order))
    try:
        for it in range(20):
            os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 0, 7, 300])))
            t, sb, db = W.random_tiny_table(rng, max_entries=10, max_numel=3000)
            C = int(rng.choice([16, 256, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"order {order} {it}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def test_walks_follow_the_alignment_of_the_side_written():
    """By default pack walks tiles of the payload where payload chunks start
    inside cache lines and unpack tiles of the receiver where receiver chunks
    do; otherwise both walk slices (plan info reports the walk taken), and
    either way the restore equals the oracle's."""
    from paper_2509_03047_amd import flashrestore as F

    names = ("FLASHRESTORE_LINE", "FLASHRESTORE_LINE_PACK", "FLASHRESTORE_LINE_UNPACK")
    old = {k: os.environ.pop(k, None) for k in names}
    rng = np.random.default_rng(77)
    try:
        table = np.zeros(3, dtype=W.TABLE_DTYPE)
        table["numel"] = [1000, 4096, 333]  # 4000, 16384, 1332 bytes
        table["dtype"] = [F.FR_F32, F.FR_F32, F.FR_F32]
        table["derive_from"] = -1
        cases = [  # src offsets, dst offsets, segment alignment, expected (pack walk, unpack walk)
            ([0, 4096, 24576], [0, 8192, 32768], 16, (4, 0)),     # payload segments inside lines
            ([0, 4096, 24576], [0, 8192, 32784], 4096, (0, 4)),   # the receiver's last entry inside a line
            ([0, 4096, 24576], [0, 8192, 32768], 4096, (0, 0)),   # every side on lines
            ([16, 4112, 24592], [16, 8208, 32784], 16, (4, 4)),
        ]
        for so, do, seg, want in cases:
            t = table.copy()
            t["src_offset"], t["dst_offset"] = so, do
            sb, db = so[-1] + 1344, do[-1] + 1344
            plan = F.Plan(t, 1024, sb, db, segment_align=seg)
            assert (plan.info["pack_walk"], plan.info["unpack_walk"]) == want, (so, do, seg)
            # the tiles the plan took are the ones a layout query predicts
            q, _, _ = F.fr_layout_query(t, 1024, sb, db, seg)
            for k in ("tile_pack", "tile_unpack", "tile_verify", "tile_checksum"):
                assert plan.info[k] == q[k], k
            del plan
            src = W.random_tiny_state(t, sb, rng)
            _check_against_oracle(t, 1024, src, sb, db, corrupt_rng=rng, seg=seg, tag=f"walks {want}")
    finally:
        for k, v in old.items():
            if v is not None:
                os.environ[k] = v


def test_mixed_tiles_per_operation():
    """Each operation with its own tile (so one plan holds several walks of
    different slice sizes) still gives the oracle's bytes."""
    names = ("FLASHRESTORE_TILE_PACK", "FLASHRESTORE_TILE_UNPACK", "FLASHRESTORE_TILE_VERIFY",
             "FLASHRESTORE_TILE_CHECKSUM")
    old = {k: os.environ.get(k) for k in names}
    rng = np.random.default_rng(91)
    try:
        for combo in ((7, 1, 3, 10), (3, 7, 10, 6), (10, 8, 7, 2)):
            for k, v in zip(names, combo):
                os.environ[k] = str(v)
            for it in range(4):
                t, sb, db = W.random_tiny_table(rng, max_entries=8, max_numel=100_000)
                C = int(rng.choice([4096, 16384, 65536]))
                src = W.random_tiny_state(t, sb, rng)
                _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng,
                                      tag=f"tiles {combo} table {it} C={C}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def test_random_midsize_tables_restore_compare_and_delta():
    """Mid-size random tables (up to 300 entries, chunks of many slices,
    derived groups, scattered layouts): whole restore and compare against the
    oracle, then a delta repair of random chunks, also against the oracle."""
    from paper_2509_03047_amd import flashrestore as F

    rng = np.random.default_rng(1234)
    for it in range(6):
        t, sb, db = W.random_tiny_table(rng, max_entries=300, max_numel=60_000)
        C = int(rng.choice([1024, 4096, 16384, 65536, 1 << 18]))
        src = W.random_tiny_state(t, sb, rng)
        log(f"midsize table {it}: {len(t)} entries, C={C}, {sb} bytes")
        _check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=f"midsize {it} C={C}")
        _delta_against_oracle(t, C, src, sb, db, rng, f"midsize {it}")


def _delta_against_oracle(t, C, src, sb, db, rng, tag):
    """Re-send a random subset of chunks into a receiver holding the oracle's
    full restore with those chunks scrambled; payload, sums, receiver and
    count must be the oracle's, and the receiver must be repaired."""
    from paper_2509_03047_amd import flashrestore as F

    plan = F.Plan(t, C, sb, db)
    n = plan.n_chunks
    if n == 0:
        return
    ids = np.sort(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False)).astype(np.uint32)
    opay, osums = cpu.pack(t, C, src)
    recv = np.full(max(db, 1), 0xA5, np.uint8)
    cpu.unpack(t, C, opay, osums, recv)
    expect = recv.copy()
    nch, base, _, _ = cpu.plan(t, C)
    for c in ids:  # scramble the listed chunks at the receiver
        k = int(np.searchsorted(base, int(c), side="right") - 1)
        j = int(c) - int(base[k])
        nb = int(t[k]["numel"]) * (4 if int(t[k]["dtype"]) == 1 else 2)
        o = int(t[k]["dst_offset"]) + j * C
        ln = min(C, nb - j * C)
        recv[o:o + ln] = rng.integers(0, 256, ln, dtype=np.uint8)
    dpay, dsums = cpu.pack_chunks(t, C, src, ids)
    g_src, g_recv = to_dev(src), to_dev(recv)
    pb = plan.delta_layout(ids)
    assert pb == dpay.size
    payload = torch.full((max(pb, 16),), 0xEE, dtype=torch.uint8, device="cuda")
    sums = torch.empty(ids.size, 2, dtype=torch.int64, device="cuda")
    bad, nbad = torch.empty((ids.size + 31) // 32, dtype=torch.int32, device="cuda"), plan.empty_counter()
    plan.pack_chunks(g_src, ids, payload, sums)
    plan.unpack_chunks(payload, sums, ids, g_recv, bad, nbad)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(payload)[:pb], dpay), f"delta payload {tag}"
    assert np.array_equal(sums_host(sums, ids.size), dsums), f"delta sums {tag}"
    orecv = recv.copy()
    obm, onbad = cpu.unpack_chunks(t, C, dpay, dsums, ids, orecv)
    assert np.array_equal(to_host(g_recv), orecv) and int(nbad.item()) == onbad == 0, f"delta {tag}"
    assert np.array_equal(orecv, expect), f"delta repair {tag}"


def test_payload_gaps_and_padding_are_never_read():
    """Unpack reads only the entries' bytes of the payload: with every gap
    byte between segments and every padding byte after a segment's last
    value overwritten, nothing is flagged and the receiver arena is the same
    as from the clean payload (the oracle reads only those bytes too)."""
    from paper_2509_03047_amd import flashrestore as F

    rng = np.random.default_rng(31)
    for it in range(20):
        t, sb, db = W.random_tiny_table(rng, max_entries=10, max_numel=3000)
        C = int(rng.choice([16, 64, 256, 4096]))
        src = W.random_tiny_state(t, sb, rng)
        r = Restore(t, C, sb, db)
        r.pack(to_dev(src) if src.size else torch.empty(16, dtype=torch.uint8, device="cuda"))
        r.unpack()
        torch.cuda.synchronize()
        clean = r.dst.clone()
        used = np.zeros(r.plan.payload_bytes, bool)
        for k in range(len(t)):
            off, _, _ = r.plan.entry_layout(k)
            nb = int(t[k]["numel"]) * (4 if int(t[k]["dtype"]) == F.FR_F32 else 2)
            if off != F.NO_PAYLOAD and nb:
                used[off:off + nb] = True
        junk = torch.from_numpy(np.where(used, 0, rng.integers(1, 256, used.size)).astype(np.uint8)).to("cuda")
        r.payload[: used.size] ^= junk  # only bytes outside the entries change
        r.dst.fill_(0xA5)
        r.unpack()
        torch.cuda.synchronize()
        assert r.bad_set() == set() and torch.equal(r.dst, clean), f"table {it} C={C}"
