"""Invariants, fault injection and brute force for the CPU oracle (CPU only).

* restore round trip: unpack(pack(x)) reproduces all four state arrays bit
  for bit when the parameters are the rounded masters, bytes outside the
  tensors are untouched, no chunk is flagged;
* the payload is the concatenation of the sent tensors with zero padding;
* single-bit faults in the donor, on the wire (payload or sums) or in a
  replica are flagged in exactly the chunks that the fault's position and the
  rounding (torch's cast) predict;
* the C oracle equals the pure-Python oracle on 1,000+ random tiny tables.
"""
import numpy as np
import pytest

from oracle import cpu, mini
from paper_2509_03047_amd import workloads as W


def _nbytes(e):
    return int(e["numel"]) * W.ESIZE[int(e["dtype"])]


def _torch_round(f32_bytes: bytes) -> bytes:
    return W._bf16_round(np.frombuffer(f32_bytes, np.float32)).tobytes()


@pytest.fixture(scope="module")
def toy():
    w = W.make_workload(0)
    src = W.fill_state(w)
    return w, src


def test_toy_sizes_closed_form(toy):
    w, src = toy
    # 3,671,296 params; 14 B of state and 12 B of payload per param, the
    # payload's 3 x 28 sent tensors back to back
    assert w.n_params == 3_671_296
    assert w.state_bytes == 14 * w.n_params == w.src_arena_bytes
    nch, base, pay, pb = cpu.plan(w.table, w.chunk_bytes)
    assert pb == 12 * w.n_params == 44_055_552
    assert int(base[-1]) == 804
    # with 4 KiB segments each sent tensor starts at a multiple of 4 KiB: the
    # five 256-element norms (1 KiB per array) leave 3 KiB gaps, except after
    # the last entry (the final norm's v, ending the payload)
    nch, base, pay, pb = cpu.plan(w.table, w.chunk_bytes, 4096)
    assert pb == 12 * w.n_params + (5 * 3 - 1) * 3072


def test_toy_round_trip(toy):
    w, src = toy
    payload, sums = cpu.pack(w.table, w.chunk_bytes, src)
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bitmap, nbad = cpu.unpack(w.table, w.chunk_bytes, payload, sums, dst)
    assert nbad == 0 and not bitmap.any()
    assert np.array_equal(dst, src)
    assert np.array_equal(cpu.checksum(w.table, w.chunk_bytes, src), sums)
    bm, nd = cpu.verify(w.table, w.chunk_bytes, src, dst)
    assert nd == 0 and not bm.any()


def test_payload_is_concatenation_with_zero_padding():
    rng = np.random.default_rng(21)
    for it in range(60):
        seg = (16, 128, 4096)[it % 3]
        t, sb, db = W.random_tiny_table(rng)
        src = W.random_tiny_state(t, sb, rng)
        payload, _ = cpu.pack(t, 64, src, seg)
        exp = bytearray()
        for e in t:
            if int(e["derive_from"]) >= 0:
                continue
            o, n = int(e["src_offset"]), _nbytes(e)
            if n:  # each non-empty segment at a multiple of seg
                exp += bytes(-len(exp) % seg)
                exp += src[o:o + n].tobytes()
        exp += bytes(-len(exp) % 16)
        assert payload.tobytes() == bytes(exp)


def test_canaries_untouched_and_round_trip_on_scattered_layouts():
    rng = np.random.default_rng(22)
    for _ in range(100):
        t, sb, db = W.random_tiny_table(rng)
        src = W.random_tiny_state(t, sb, rng)
        C = int(rng.choice([16, 32, 64, 256]))
        payload, sums = cpu.pack(t, C, src)
        dst = np.full(db + 64, 0xA5, np.uint8)
        bm, nbad = cpu.unpack(t, C, payload, sums, dst)
        assert nbad == 0
        covered = np.zeros(dst.size, bool)
        for e in t:
            so, do, n = int(e["src_offset"]), int(e["dst_offset"]), _nbytes(e)
            assert np.array_equal(dst[do:do + n], src[so:so + n])
            covered[do:do + n] = True
        assert (dst[~covered] == 0xA5).all()


def _chunk_of(t, C, k, byte):
    _, base, _, _ = mini.plan(t, C)
    return base[k] + byte // C


def _state_table_small():
    tensors = [("a", 40), ("b", 3), ("c", 17)]
    t, nb = W.state_table(tensors)
    return t, nb


def test_flip_in_payload_flags_predicted_chunks():
    t, nb = _state_table_small()
    rng = np.random.default_rng(23)
    src = W.random_tiny_state(t, nb, rng)
    C = 32
    payload, sums = cpu.pack(t, C, src)
    _, base, pay, _ = mini.plan(t, C)
    nc = base[-1]
    seg = []  # (entry, payload start, nbytes) of sent entries
    for k, e in enumerate(t):
        if pay[k] is not None:
            seg.append((k, pay[k], _nbytes(e)))
    derived_of = {int(e["derive_from"]): k for k, e in enumerate(t) if int(e["derive_from"]) >= 0}
    for bit in range(payload.size * 8):
        p = payload.copy()
        p[bit // 8] ^= np.uint8(1 << (bit % 8))
        dst = np.zeros(nb, np.uint8)
        bm, nbad = cpu.unpack(t, C, p, sums, dst)
        got = set(cpu.bitmap_to_set(bm, nc))
        exp = set()
        for k, start, n in seg:
            off = bit // 8 - start
            if 0 <= off < n:
                exp.add(_chunk_of(t, C, k, off))
                if k in derived_of:  # master on the wire: its bf16 image may change
                    d = derived_of[k]
                    el = off // 4
                    mb = p[start + 4 * el:start + 4 * el + 4].tobytes()
                    so = int(t[d]["src_offset"])
                    if _torch_round(mb) != src[so + 2 * el:so + 2 * el + 2].tobytes():
                        exp.add(_chunk_of(t, C, d, 2 * el))
        assert got == exp, bit
        assert nbad == len(exp)


def test_flip_in_sums_flags_that_chunk():
    t, nb = _state_table_small()
    rng = np.random.default_rng(24)
    src = W.random_tiny_state(t, nb, rng)
    C = 64
    payload, sums = cpu.pack(t, C, src)
    nc = sums.size // 2
    for c in range(nc):
        for word in (0, 1):
            for bit in (0, 17, 63):
                s = sums.copy()
                s[2 * c + word] ^= np.uint64(1 << bit)
                dst = np.zeros(nb, np.uint8)
                bm, nbad = cpu.unpack(t, C, payload, s, dst)
                assert cpu.bitmap_to_set(bm, nc) == [c] and nbad == 1


def test_flip_in_sender_state_before_pack():
    """A flipped bf16 param is flagged (the receiver re-derives it from the
    master); a flipped master is sent consistently and flags only the derived
    param chunk, and only when its rounding changes."""
    t, nb = _state_table_small()
    rng = np.random.default_rng(25)
    src = W.random_tiny_state(t, nb, rng)
    C = 16
    nc = mini.plan(t, C)[1][-1]
    for k, e in enumerate(t):
        n = _nbytes(e)
        o = int(e["src_offset"])
        for byte in range(n):
            for bit in (0, 7):
                s = src.copy()
                s[o + byte] ^= np.uint8(1 << bit)
                payload, sums = cpu.pack(t, C, s)
                dst = np.zeros(nb, np.uint8)
                bm, _ = cpu.unpack(t, C, payload, sums, dst)
                got = set(cpu.bitmap_to_set(bm, nc))
                if int(e["derive_from"]) >= 0:
                    exp = {_chunk_of(t, C, k, byte)}
                else:
                    exp = set()
                    for d, ed in enumerate(t):
                        if int(ed["derive_from"]) == k:
                            el = byte // 4
                            new = _torch_round(s[o + 4 * el:o + 4 * el + 4].tobytes())
                            od = int(ed["src_offset"])
                            if new != src[od + 2 * el:od + 2 * el + 2].tobytes():
                                exp.add(_chunk_of(t, C, d, 2 * el))
                assert got == exp, (k, byte, bit)


def test_verify_replicas_locates_flips_closed_form():
    w = W.make_workload(0)
    a = W.fill_state(w)
    nc = cpu.n_chunks(w.table, w.chunk_bytes)
    # position p (byte) -> chunk id: entries are contiguous in table order
    starts = w.table["src_offset"].astype(np.int64)
    for k in (0, 1, 64, 4096):
        b = a.copy()
        pos = W.flip_positions(a.size * 8, k, 4000 + k)
        W.apply_flips(b, pos)
        exp = set()
        for p in pos:
            byte = int(p) // 8
            e = int(np.searchsorted(starts, byte, side="right") - 1)
            exp.add(_chunk_of(w.table, w.chunk_bytes, e, byte - int(starts[e])))
        bm, nd = cpu.verify(w.table, w.chunk_bytes, a, b)
        assert set(cpu.bitmap_to_set(bm, nc)) == exp
        assert nd == len(exp)
        # the chunk sums see the same set on this input
        _, _, sa, sb = cpu.verify(w.table, w.chunk_bytes, a, b, with_sums=True)
        sdiff = {c for c in range(nc) if tuple(sa[2 * c:2 * c + 2]) != tuple(sb[2 * c:2 * c + 2])}
        assert sdiff == exp


@pytest.mark.slow
def test_c_oracle_equals_python_oracle_bruteforce():
    rng = np.random.default_rng(26)
    n_tables = 1000
    for it in range(n_tables):
        t, sb, db = W.random_tiny_table(rng, max_numel=120 if it % 4 else 300)
        C = int(rng.choice([16, 32, 64, 256]))
        src = W.random_tiny_state(t, sb, rng)
        payload, sums = cpu.pack(t, C, src)
        mp, ms = mini.pack(t, C, src.tobytes())
        assert payload.tobytes() == mp
        assert [tuple(int(x) for x in sums[2 * i:2 * i + 2]) for i in range(len(ms))] == ms
        # corrupt a random payload bit half of the time
        p = payload.copy()
        if p.size and rng.random() < 0.5:
            b = int(rng.integers(0, p.size * 8))
            p[b // 8] ^= np.uint8(1 << (b % 8))
        dst = np.full(db, 0xA5, np.uint8)
        bm, nbad = cpu.unpack(t, C, p, sums, dst)
        mdst = bytearray(np.full(db, 0xA5, np.uint8).tobytes())
        mbad = mini.unpack(t, C, p.tobytes(), ms, mdst)
        assert dst.tobytes() == bytes(mdst)
        assert set(cpu.bitmap_to_set(bm, len(ms))) == mbad and nbad == len(mbad)
        b2 = src.copy()
        if b2.size:
            for _ in range(int(rng.integers(0, 3))):
                b = int(rng.integers(0, b2.size * 8))
                b2[b // 8] ^= np.uint8(1 << (b % 8))
        vb, nd = cpu.verify(t, C, src, b2)
        assert set(cpu.bitmap_to_set(vb, len(ms))) == mini.verify(t, C, src.tobytes(), b2.tobytes())
