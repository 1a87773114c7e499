"""Pins of the CPU oracle against values fixed outside it (CPU only).

Every part of the oracle's arithmetic is checked against something other
than itself: hand-worked values (tests/golden), closed forms, library
routines (numpy's modular integer sums, torch's bf16 cast), exhaustive
enumeration and detection properties that a dropped term, a wrong index or
a swapped byte order would break.
"""
import os

import numpy as np
import pytest
import torch

from oracle import cpu, mini

M64 = (1 << 64) - 1


def _golden_frsum(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "frsum_worked.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            p = line.split()
            if p[0] == "hex":
                data = bytes.fromhex(p[1])
                s, ws = int(p[2]), int(p[3])
            else:
                data = bytes([int(p[1], 16)]) * int(p[2])
                s, ws = int(p[3]), int(p[4])
            rows.append((data, s, ws))
    return rows


def _golden_rne(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "rne_bf16_special.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            p = line.split()
            rows.append((int(p[0], 16), int(p[1], 16)))
    return rows


def test_frsum_worked_values(golden_dir):
    rows = _golden_frsum(golden_dir)
    assert len(rows) >= 8
    for data, s, ws in rows:
        assert cpu.frsum(data) == (s, ws), data[:16].hex()
        if len(data) <= 4096:
            assert mini.frsum(data) == (s, ws)


def test_frsum_matches_numpy_modular_sums():
    """sum = numpy uint64 sum of the words; wsum = numpy uint64 dot with 1..n
    (numpy's uint64 arithmetic wraps mod 2^64)."""
    rng = np.random.default_rng(11)
    for n_words in (1, 3, 64, 1000, 100_000):
        w = rng.integers(0, 1 << 32, size=n_words, dtype=np.uint64)
        b = w.astype("<u4").tobytes()
        with np.errstate(over="ignore"):
            s = int(np.sum(w, dtype=np.uint64))
            ws = int(np.sum(w * np.arange(1, n_words + 1, dtype=np.uint64), dtype=np.uint64))
        assert cpu.frsum(b) == (s, ws)


def test_frsum_shift_law():
    """Prefixing k zero words leaves sum and adds k*sum to wsum (mod 2^64);
    catches an off-by-one or dropped word index."""
    rng = np.random.default_rng(12)
    x = rng.integers(0, 256, size=1000, dtype=np.uint8).tobytes()
    s, ws = cpu.frsum(x)
    for k in (1, 5, 4096):
        s2, ws2 = cpu.frsum(bytes(4 * k) + x)
        assert s2 == s and ws2 == (ws + k * s) & M64


def test_frsum_all_ones_closed_form():
    for n in (1, 2, 16384, 92681, 92682, 131072):
        b = b"\xff" * (4 * n)
        exp = ((n * 0xFFFFFFFF) & M64, (0xFFFFFFFF * n * (n + 1) // 2) & M64)
        assert cpu.frsum(b) == exp, n


def test_frsum_bf16_tail_is_zero_filled():
    """A chunk of 2 mod 4 bytes sums as if two zero bytes followed."""
    rng = np.random.default_rng(13)
    for n in (2, 6, 30, 1022):
        x = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        assert cpu.frsum(x) == cpu.frsum(x + b"\0\0")
        assert mini.frsum(x) == cpu.frsum(x)


def test_frsum_detects_every_single_flip_exhaustive():
    rng = np.random.default_rng(14)
    base = rng.integers(0, 256, size=64, dtype=np.uint8)
    ref = cpu.frsum(base)
    for bit in range(64 * 8):
        v = base.copy()
        v[bit // 8] ^= np.uint8(1 << (bit % 8))
        s, _ = cpu.frsum(v)
        assert s != ref[0], bit


def test_frsum_detects_every_double_flip_exhaustive():
    """All 130,816 pairs of distinct bits in a 64-byte chunk change (sum, wsum)."""
    rng = np.random.default_rng(15)
    base = rng.integers(0, 256, size=64, dtype=np.uint8)
    ref = cpu.frsum(base)
    bits = 64 * 8
    count = 0
    for a in range(bits):
        va = base.copy()
        va[a // 8] ^= np.uint8(1 << (a % 8))
        for b in range(a + 1, bits):
            v = va.copy()
            v[b // 8] ^= np.uint8(1 << (b % 8))
            assert cpu.frsum(v) != ref, (a, b)
            count += 1
    assert count == bits * (bits - 1) // 2 == 130816


def test_frsum_detects_word_swaps():
    rng = np.random.default_rng(16)
    w = rng.integers(0, 1 << 32, size=32, dtype=np.uint64).astype("<u4")
    ref = cpu.frsum(w.tobytes())
    for i in range(32):
        for j in range(i + 1, 32):
            if w[i] == w[j]:
                continue
            v = w.copy()
            v[i], v[j] = w[j], w[i]
            s, ws = cpu.frsum(v.tobytes())
            assert s == ref[0] and ws != ref[1]


def test_rne_special_values(golden_dir):
    rows = _golden_rne(golden_dir)
    assert len(rows) >= 20
    for u, h in rows:
        assert cpu.rne_bf16(u) == h, hex(u)
        assert mini.rne_bf16(u) == h, hex(u)


def _torch_bf16(u32):
    return torch.from_numpy(u32.view(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


@pytest.mark.slow
def test_rne_exhaustive_vs_torch_cast():
    """All 2^32 fp32 patterns: the oracle's nearest-neighbour rounding equals
    torch's CPU bf16 cast on every non-NaN input; NaNs follow the reading."""
    block = 1 << 26
    for start in range(0, 1 << 32, block):
        u = np.arange(start, start + block, dtype=np.uint64).astype(np.uint32)
        got = cpu.rne_bf16_array(u)
        nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        ref = _torch_bf16(u)
        ok = (got == ref) | nan
        assert ok.all(), hex(int(u[np.argmin(ok)]))
        if nan.any():
            exp_nan = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
            assert (got[nan] == exp_nan).all()


def test_rne_properties():
    rng = np.random.default_rng(17)
    # values already representable in bf16 are returned unchanged
    h = rng.integers(0, 1 << 16, size=100_000, dtype=np.uint64).astype(np.uint32)
    h = h[((h & 0x7FFF) <= 0x7F80)]
    assert (cpu.rne_bf16_array(h << np.uint32(16)) == h.astype(np.uint16)).all()
    # monotone on positive finite inputs
    u = np.sort(rng.integers(0, 0x7F800000, size=200_000, dtype=np.uint64)).astype(np.uint32)
    r = cpu.rne_bf16_array(u)
    assert (np.diff(r.astype(np.int64)) >= 0).all()
    # sign symmetry
    assert (cpu.rne_bf16_array(u | np.uint32(0x80000000)) == (r | np.uint16(0x8000))).all()


def test_rne_mini_agrees_on_random_patterns():
    rng = np.random.default_rng(18)
    u = rng.integers(0, 1 << 32, size=3000, dtype=np.uint64).astype(np.uint32)
    got = cpu.rne_bf16_array(u)
    for x, g in zip(u, got):
        assert mini.rne_bf16(int(x)) == int(g)


@pytest.mark.parametrize("name", ["pack_worked.txt", "pack_worked_packed.txt"])
def test_pack_worked_example(golden_dir, name):
    """A three-entry pack worked by hand (tests/golden/pack_worked*.txt, with
    4 KiB and 16-byte payload segments): payload bytes, segment placement,
    zero gaps and every chunk's sums, for both oracles; the restore of it
    reproduces the arena."""
    from paper_2509_03047_amd import workloads as W

    rows, src, segs, sums, C, ab, pb, deltas, seg = [], {}, {}, [], 0, 0, 0, [], 0
    with open(os.path.join(golden_dir, name)) as f:
        for line in f:
            p = line.split()
            if not p or p[0].startswith("#"):
                continue
            if p[0] == "entry":
                rows.append(tuple(int(x) for x in p[1:]))
            elif p[0] == "chunk_bytes":
                C = int(p[1])
            elif p[0] == "segment_align":
                seg = int(p[1])
            elif p[0] == "arena_bytes":
                ab = int(p[1])
            elif p[0] == "src":
                src[int(p[1])] = bytes.fromhex(p[2])
            elif p[0] == "payload_bytes":
                pb = int(p[1])
            elif p[0] == "segment":
                segs[int(p[1])] = bytes.fromhex(p[2])
            elif p[0] == "sums":
                sums += [int(p[1]), int(p[2])]
            elif p[0] == "delta":
                deltas.append(([int(x) for x in p[1].split(",")],
                               [None if x == "-" else int(x) for x in p[2].split(",")], int(p[3])))
    t = np.array(rows, dtype=W.TABLE_DTYPE)
    arena = np.zeros(ab, np.uint8)
    for o, b in src.items():
        arena[o:o + len(b)] = np.frombuffer(b, np.uint8)
    expect = np.zeros(pb, np.uint8)
    for o, b in segs.items():
        expect[o:o + len(b)] = np.frombuffer(b, np.uint8)
    assert seg in (16, 4096)
    pay, s = cpu.pack(t, C, arena, seg)
    assert np.array_equal(pay, expect) and [int(x) for x in s] == sums
    mp, ms = mini.pack(t, C, arena.tobytes(), seg)
    assert mp == expect.tobytes() and [x for pair in ms for x in pair] == sums
    dst = np.zeros(ab, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, s, dst, seg)
    assert nbad == 0 and np.array_equal(dst, arena)
    # delta lists: offsets, sizes, and the bytes at those offsets
    assert len(deltas) == 4
    for ids, offs, size in deltas:
        ia = np.array(ids, np.uint32)
        off, got_size = cpu.delta_layout(t, C, ia, seg)
        assert got_size == size and [None if o == cpu.NO_PAYLOAD else int(o) for o in off] == offs
        dp, ds = cpu.pack_chunks(t, C, arena, ia, seg)
        assert dp.size == size and [int(x) for x in ds] == [v for c in ids for v in sums[2 * c:2 * c + 2]]
        _, base, _, _ = cpu.plan(t, C, seg)
        for c, o in zip(ids, offs):
            if o is None:
                continue
            k = int(np.searchsorted(base, c, side="right") - 1)
            so = int(t[k]["src_offset"]) + (c - int(base[k])) * C
            ln = min(C, int(t[k]["numel"]) * (4 if int(t[k]["dtype"]) == 1 else 2) - (c - int(base[k])) * C)
            assert np.array_equal(dp[o:o + ln], arena[so:so + ln])
