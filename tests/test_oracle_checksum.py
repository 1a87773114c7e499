"""Pins of the oracle's checksum paths (CPU only): the checksum of one
replica, the replica compare's sums of both arenas, and the checksum of a
list of chunks.

A healthy replica's chunk sums are what the donor sends with its state
(Section III-E: the recreated process must end up holding the replica's
state), so each of these must equal the sums a pack of the same arena
produces, read at the sender offsets.  Pinned here by:
* a hand-worked table whose sender and receiver offsets differ and whose
  bytes at the two differ, with empty entries at the start, in the middle
  and at the end (tests/golden/checksum_worked.txt);
* 240 random tiny tables with independent sender and receiver layouts and
  empty entries inserted at the start, in the middle and at the end: the C
  oracle's checksum, compare sums and chunk-list checksum equal the sums of
  the pure-Python oracle's pack, at every chunk id next to an empty entry,
  the first and the last chunk included;
* location: a single flipped bit of the arena changes the sums of exactly
  the chunk that holds it, found by walking the table in the test;
* the consistency check from sums alone (both oracles): replicas built from
  FRSUM's definition to differ in sum alone, in wsum alone, or in one bit of
  the last chunk are flagged exactly there, identical ones not at all,
  single flips at the chunks that hold them, and the C oracle's bitmap has
  its words and ragged last word right for every count from 0 to 100.
"""
import os

import numpy as np
import pytest

from oracle import cpu, mini
from paper_2509_03047_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))


def load_checksum_golden(path=None):
    """The worked example: (table, C, arena A, sums, list ids, list sums,
    arena B, diff set, sums of B)."""
    path = path or os.path.join(HERE, "golden", "checksum_worked.txt")
    rows, arena, sums, sums_b = [], None, [], []
    C = n = ids = flip = diff = None
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *v = line.split()
            if key == "entry":
                rows.append(tuple(int(x) for x in v))
            elif key == "chunk_bytes":
                C = int(v[0])
            elif key == "arena_bytes":
                n = int(v[0])
                arena = np.zeros(n, np.uint8)
            elif key == "arena":
                b = bytes.fromhex(v[1])
                arena[int(v[0]):int(v[0]) + len(b)] = np.frombuffer(b, np.uint8)
            elif key == "sums":
                sums.append((int(v[0]), int(v[1])))
            elif key == "list":
                ids = [int(x) for x in v[0].split(",")]
            elif key == "flip":
                flip = (int(v[0]), int(v[1]))
            elif key == "diff":
                diff = {int(x) for x in v[0].split(",")}
            elif key == "sums_b":
                sums_b.append((int(v[0]), int(v[1])))
    t = np.zeros(len(rows), W.TABLE_DTYPE)
    for k, (so, do, ne, dt, der) in enumerate(rows):
        t[k] = (so, do, ne, dt, der)
    b = arena.copy()
    b[flip[0]] ^= np.uint8(1 << flip[1])
    return t, C, arena, sums, ids, [sums[i] for i in ids], b, diff, sums_b


def _pairs(flat):
    flat = np.asarray(flat, np.uint64)
    return [(int(flat[2 * i]), int(flat[2 * i + 1])) for i in range(flat.size // 2)]


def test_golden_is_a_scattered_layout():
    t, C, a, *_ = load_checksum_golden()
    nb = t["numel"] * np.where(t["dtype"] == 1, 4, 2)
    live = nb > 0
    # sender and receiver offsets differ, and so do the bytes found there
    assert (t["src_offset"][live] != t["dst_offset"][live]).all()
    for e in t[live]:
        k = int(e["numel"]) * (4 if int(e["dtype"]) == 1 else 2)
        s, d = int(e["src_offset"]), int(e["dst_offset"])
        assert a[s:s + k].tobytes() != a[d:d + k].tobytes()
    assert nb[0] == 0 and nb[-1] == 0 and (nb[1:-1] == 0).any()


def test_c_oracle_checksum_paths_on_the_worked_table():
    t, C, a, sums, ids, list_sums, b, diff, sums_b = load_checksum_golden()
    assert _pairs(cpu.checksum(t, C, a)) == sums
    bm, nd, sa, sb = cpu.verify(t, C, a, b, with_sums=True)
    assert set(cpu.bitmap_to_set(bm, len(sums))) == diff and nd == len(diff)
    assert _pairs(sa) == sums and _pairs(sb) == sums_b
    assert _pairs(cpu.checksum_chunks(t, C, a, np.array(ids))) == list_sums
    # the pack of the same arena sends the same sums
    assert _pairs(cpu.pack(t, C, a)[1]) == sums


def test_python_oracle_checksum_paths_on_the_worked_table():
    t, C, a, sums, ids, list_sums, b, diff, sums_b = load_checksum_golden()
    ab, bb = a.tobytes(), b.tobytes()
    assert mini.checksum(t, C, ab) == sums
    d, sa, sb = mini.verify_with_sums(t, C, ab, bb)
    assert d == diff and sa == sums and sb == sums_b
    assert mini.checksum_chunks(t, C, ab, ids) == list_sums
    assert mini.pack(t, C, ab)[1] == sums


def with_empty_entries(t, sb, db, rng):
    """The table with empty entries inserted at the start, at a random
    position inside and at the end (derive_from indices remapped); their
    offsets are random multiples of 16 inside the arenas."""
    n = len(t)
    mid = int(rng.integers(1, n + 1)) if n else 0
    at = [0, mid, n]  # insert before old index 0, before old index mid, after the last
    out = np.zeros(n + 3, W.TABLE_DTYPE)
    pos, newpos = 0, []
    for i in range(n + 1):
        while pos < 3 and at[pos] == i:
            e = out[i + pos]
            e["src_offset"] = 16 * int(rng.integers(0, sb // 16 + 1))
            e["dst_offset"] = 16 * int(rng.integers(0, db // 16 + 1))
            e["numel"] = 0
            e["dtype"] = int(rng.choice([W.F32, W.BF16]))
            e["derive_from"] = -1
            pos += 1
        if i < n:
            newpos.append(i + pos)
            out[i + pos] = t[i]
    for i in range(n):
        d = int(t[i]["derive_from"])
        if d >= 0:
            out[newpos[i]]["derive_from"] = newpos[d]
    return out


def _edge_ids(t, C):
    """Chunk ids next to empty entries (the last chunk before, the first
    after), plus the first and the last chunk."""
    _, base, _, _ = cpu.plan(t, C)
    base = [int(x) for x in base]
    n = base[-1]
    ids = {0, n - 1} if n else set()
    for k in range(len(t)):
        if base[k] == base[k + 1]:  # empty entry k
            if base[k] > 0:
                ids.add(base[k] - 1)
            if base[k] < n:
                ids.add(base[k])
    return sorted(ids)


def _chunk_of_byte(t, C, p):
    """Global chunk holding arena byte p at the sender offsets (walking the
    table), or None.  Sender ranges of these tables do not overlap."""
    c = 0
    for e in t:
        nb = int(e["numel"]) * (4 if int(e["dtype"]) == 1 else 2)
        o = int(e["src_offset"])
        if o <= p < o + nb:
            return c + (p - o) // C
        c += -(-nb // C)
    return None


def test_checksum_paths_equal_the_pack_sums_on_scattered_tables():
    rng = np.random.default_rng(2024)
    n_edge = 0
    for it in range(240):
        t0, sb, db = W.random_tiny_table(rng, max_entries=6, max_numel=200)
        t = with_empty_entries(t0, sb, db, rng)
        assert (t["numel"][[0, -1]] == 0).all()
        C = int(rng.choice([8, 16, 32, 64, 256]))
        a = W.random_tiny_state(t, sb, rng)
        b = a.copy()
        for _ in range(int(rng.integers(0, 4))):
            if sb:
                p = int(rng.integers(0, sb * 8))
                b[p // 8] ^= np.uint8(1 << (p % 8))
        want_a = mini.pack(t, C, a.tobytes())[1]
        want_b = mini.pack(t, C, b.tobytes())[1]
        n = len(want_a)
        assert _pairs(cpu.checksum(t, C, a)) == want_a, it
        bm, nd, sa, sbs = cpu.verify(t, C, a, b, with_sums=True)
        assert _pairs(sa) == want_a and _pairs(sbs) == want_b, it
        assert set(cpu.bitmap_to_set(bm, n)) == mini.verify(t, C, a.tobytes(), b.tobytes()), it
        edge = _edge_ids(t, C)
        n_edge += len(edge)
        extra = list(rng.integers(0, n, size=5)) if n else []
        ids = np.array(edge + [int(x) for x in extra], np.uint64)
        rng.shuffle(ids)
        got = _pairs(cpu.checksum_chunks(t, C, a, ids))
        assert got == [want_a[int(i)] for i in ids], it
        assert mini.checksum_chunks(t, C, a.tobytes(), [int(i) for i in ids]) == got, it
    assert n_edge > 500  # chunks next to empty entries were exercised


def test_a_flipped_bit_changes_only_its_chunk():
    rng = np.random.default_rng(77)
    for it in range(60):
        t0, sb, db = W.random_tiny_table(rng, max_entries=5, max_numel=150)
        t = with_empty_entries(t0, sb, db, rng)
        C = int(rng.choice([16, 32, 64]))
        a = W.random_tiny_state(t, sb, rng)
        ref = _pairs(cpu.checksum(t, C, a))
        for _ in range(8):
            if not sb:
                break
            p = int(rng.integers(0, sb))
            b = a.copy()
            b[p] ^= np.uint8(1 << int(rng.integers(0, 8)))
            got = _pairs(cpu.checksum(t, C, b))
            changed = {c for c, (x, y) in enumerate(zip(ref, got)) if x != y}
            c = _chunk_of_byte(t, C, p)
            assert changed == (set() if c is None else {c}), (it, p)


# ------------------------------------------------ consistency from sums alone

def _crafted_sums_cases():
    """One fp32 entry of 64 words in 64-byte chunks (4 chunks of 16 words),
    and replicas that differ in one chunk only in (a) sum alone, (b) wsum
    alone, (c) a single bit of the last chunk, built from FRSUM's
    definition: words w_i, w_j of chunk 2 with bit q set in w_j and clear in
    w_i.  (a) w_0 gains bit q + 1 and w_1 loses bit q: sum +2^q, wsum
    1 * 2^(q+1) - 2 * 2^q = 0.  (b) w_0 gains bit q and w_1 loses it: sum
    unchanged, wsum 2^q (1 - 2) != 0."""
    t = np.zeros(1, dtype=W.TABLE_DTYPE)
    t["numel"], t["dtype"], t["derive_from"] = 64, W.F32, -1
    a = np.zeros(256, np.uint8)
    words = a.view("<u4")
    words[:] = np.arange(64, dtype=np.uint32) * np.uint32(2654435761)
    q = 5
    w0, w1 = 32, 33  # words 0 and 1 of chunk 2
    words[w0] &= ~np.uint32((1 << q) | (1 << (q + 1)))
    words[w1] |= np.uint32(1 << q)
    cases = []
    b = a.copy()
    bw = b.view("<u4")
    bw[w0] |= np.uint32(1 << (q + 1))
    bw[w1] &= ~np.uint32(1 << q)
    cases.append(("sum only", b, {2}))
    b = a.copy()
    bw = b.view("<u4")
    bw[w0] |= np.uint32(1 << q)
    bw[w1] &= ~np.uint32(1 << q)
    cases.append(("wsum only", b, {2}))
    b = a.copy()
    b[255] ^= np.uint8(0x80)
    cases.append(("last chunk", b, {3}))
    cases.append(("identical", a.copy(), set()))
    return t, 64, a, cases


def compare_pins(compare, checksum):
    """Names of the pins that `compare(sums_a, sums_b) -> set` fails, with
    `checksum(table, C, arena bytes) -> [(sum, wsum), ...]` giving each
    replica's sums."""
    failed = []
    t, C, a, cases = _crafted_sums_cases()
    sa = checksum(t, C, a.tobytes())
    for name, b, want in cases:
        sb = checksum(t, C, b.tobytes())
        if name == "sum only" and not (sa[2][0] != sb[2][0] and sa[2][1] == sb[2][1]):
            failed.append("construction (sum only)")
        if name == "wsum only" and not (sa[2][0] == sb[2][0] and sa[2][1] != sb[2][1]):
            failed.append("construction (wsum only)")
        if compare(sa, sb) != want:
            failed.append(name)
    rng = np.random.default_rng(77)
    for _ in range(60):  # single flips land in the chunks that hold them
        t0, sb_, db = W.random_tiny_table(rng, max_entries=6, max_numel=200)
        if sb_ == 0:
            continue
        C = int(rng.choice([16, 32, 64, 256]))
        x = W.random_tiny_state(t0, sb_, rng)
        y = x.copy()
        want = set()
        for p in rng.integers(0, sb_, size=int(rng.integers(1, 4))):
            y[p] ^= np.uint8(1 << int(rng.integers(0, 8)))
            c = _chunk_of_byte(t0, C, int(p))
            if c is not None:
                want.add(c)
        if compare(checksum(t0, C, x.tobytes()), checksum(t0, C, y.tobytes())) != want:
            failed.append("flip locations")
            break
    return failed


def _c_compare(sa, sb):
    bm, nd = cpu.compare_sums(np.asarray(sa, np.uint64).reshape(-1), np.asarray(sb, np.uint64).reshape(-1))
    got = set(cpu.bitmap_to_set(bm, len(sa)))
    assert nd == len(got)
    return got


def test_compare_sums_pins_accept_both_oracles():
    assert compare_pins(_c_compare, lambda t, C, x: _pairs(cpu.checksum(t, C, np.frombuffer(x, np.uint8)))) == []
    assert compare_pins(mini.compare_sums, mini.checksum) == []


def test_c_compare_sums_bitmap_words_and_ragged_counts():
    """Bits past the last chunk stay clear; every count from 0 to 100 chunks
    (ragged last words) against the pure-Python oracle."""
    rng = np.random.default_rng(5)
    for n in range(0, 101):
        a = rng.integers(0, 4, size=2 * n, dtype=np.uint64)
        b = a.copy()
        sel = rng.random(2 * n) < 0.2
        b[sel] ^= np.uint64(1)
        bm, nd = cpu.compare_sums(a, b)
        assert bm.size == (n + 31) // 32
        want = mini.compare_sums(_pairs(a), _pairs(b))
        assert set(cpu.bitmap_to_set(bm, n)) == want and nd == len(want)
        if n % 32:
            assert int(bm[-1]) >> (n % 32) == 0
