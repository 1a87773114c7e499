"""Second oracle, pure Python, for tiny inputs.  TEST INFRASTRUCTURE ONLY.

Same definitions as the C oracle, written independently: Python integers
for the modular sums, exact rationals (``fractions.Fraction``) for rounding,
byte strings for arenas.  Used to cross-check the C oracle by brute force
on many random tiny tables.
"""
from __future__ import annotations

from fractions import Fraction

M64 = (1 << 64) - 1
SEGMENT = 16  # default: a payload segment starts at a multiple of this


def _up(x, a):
    return -(-x // a) * a


def frsum(b: bytes):
    """(sum, wsum) of little-endian 32-bit words, zero-filled tail."""
    s = ws = 0
    for i in range(0, len(b), 4):
        w = int.from_bytes(b[i:i + 4].ljust(4, b"\0"), "little")
        s += w
        ws += (i // 4 + 1) * w
    return s & M64, ws & M64


def _f32_value(u: int) -> Fraction:
    """Exact value of a finite fp32 bit pattern's magnitude."""
    e = (u >> 23) & 0xFF
    m = u & 0x7FFFFF
    if e == 0:
        return Fraction(m, 1 << 149)
    return Fraction((1 << 23) | m, 1 << 23) * (Fraction(2) ** (e - 127))


def _bf16_value(h: int) -> Fraction:
    h &= 0x7FFF
    if h == 0x7F80:
        return Fraction(2) ** 128  # one step past the largest finite value
    return _f32_value(h << 16)


def rne_bf16(u: int) -> int:
    u &= 0xFFFFFFFF
    mag, sign = u & 0x7FFFFFFF, (u >> 16) & 0x8000
    if mag > 0x7F800000:
        return (u >> 16) | 0x0040
    if mag == 0x7F800000:
        return sign | 0x7F80
    x = _f32_value(mag)
    cands = [mag >> 16, (mag >> 16) + 1]
    best = min(cands, key=lambda h: (abs(_bf16_value(h) - x), h & 1))
    return sign | best


def _esize(dt):
    return 4 if dt == 1 else 2


def plan(table, C, seg=SEGMENT):
    nch, base, pay = [], [0], []
    end = 0
    for e in table:
        nb = int(e["numel"]) * _esize(int(e["dtype"]))
        nch.append(-(-nb // C))
        base.append(base[-1] + nch[-1])
        if int(e["derive_from"]) >= 0:
            pay.append(None)
        elif nb == 0:
            pay.append(_up(end, 16))  # an empty entry occupies no segment
        else:
            pay.append(_up(end, seg))
            end = pay[-1] + nb
    return nch, base, pay, _up(end, 16)


def _chunks(table, C, arena: bytes, key):
    """Yield (global id, bytes) of every chunk, reading entries at ``key``."""
    c = 0
    for e in table:
        nb = int(e["numel"]) * _esize(int(e["dtype"]))
        o = int(e[key])
        for j in range(0, nb, C):
            yield c, arena[o + j:o + min(j + C, nb)]
            c += 1


def pack(table, C, src: bytes, seg=SEGMENT):
    _, base, pay, pb = plan(table, C, seg)
    payload = bytearray(pb)
    for k, e in enumerate(table):
        if pay[k] is not None:
            nb = int(e["numel"]) * _esize(int(e["dtype"]))
            o = int(e["src_offset"])
            payload[pay[k]:pay[k] + nb] = src[o:o + nb]
    sums = [frsum(b) for _, b in _chunks(table, C, src, "src_offset")]
    return bytes(payload), sums


def unpack(table, C, payload: bytes, sums, dst: bytearray, seg=SEGMENT):
    _, base, pay, _ = plan(table, C, seg)
    for k, e in enumerate(table):
        nb = int(e["numel"]) * _esize(int(e["dtype"]))
        o = int(e["dst_offset"])
        s = int(e["derive_from"])
        if s < 0:
            dst[o:o + nb] = payload[pay[k]:pay[k] + nb]
        else:
            for i in range(int(e["numel"])):
                u = int.from_bytes(payload[pay[s] + 4 * i:pay[s] + 4 * i + 4], "little")
                dst[o + 2 * i:o + 2 * i + 2] = rne_bf16(u).to_bytes(2, "little")
    got = [frsum(b) for _, b in _chunks(table, C, bytes(dst), "dst_offset")]
    bad = {c for c, (g, w) in enumerate(zip(got, sums)) if tuple(g) != tuple(w)}
    return bad


def verify(table, C, a: bytes, b: bytes):
    ca = dict(_chunks(table, C, a, "src_offset"))
    cb = dict(_chunks(table, C, b, "src_offset"))
    return {c for c in ca if ca[c] != cb[c]}


def checksum(table, C, arena: bytes):
    """FRSUM of every chunk of one replica's arena, read at the sender
    offsets: what a healthy replica would send for each chunk."""
    return [frsum(b) for _, b in _chunks(table, C, arena, "src_offset")]


def compare_sums(sums_a, sums_b):
    """Chunks whose sums differ between two replicas' checksums (each a
    list of (sum, wsum) per chunk): the consistency check that needs only
    the sums to travel."""
    return {c for c, (x, y) in enumerate(zip(sums_a, sums_b)) if tuple(x) != tuple(y)}


def verify_with_sums(table, C, a: bytes, b: bytes):
    """The replica compare together with both arenas' chunk sums."""
    return verify(table, C, a, b), checksum(table, C, a), checksum(table, C, b)


def _entry_of(base, c):
    """Entry k with base[k] <= c < base[k + 1] (base: prefix of chunk counts,
    n + 1 values); empty entries (base[k] == base[k + 1]) hold no chunk, so
    the search takes the last entry whose first chunk is <= c."""
    lo, hi = 0, len(base) - 1
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if base[mid] <= c:
            lo = mid
        else:
            hi = mid
    return lo


def checksum_chunks(table, C, arena: bytes, ids):
    """FRSUM of the listed chunks (global ids, any order) at sender offsets."""
    _, base, _, _ = plan(table, C)
    out = []
    for c in ids:
        k = _entry_of(base, int(c))
        o, ln = _chunk_bytes(table, C, k, int(c) - base[k], arena, "src_offset")
        out.append(frsum(arena[o:o + ln]))
    return out


def _chunk_map(table, C):
    """Global chunk id -> (entry, index within entry)."""
    out = []
    for k, e in enumerate(table):
        nb = int(e["numel"]) * _esize(int(e["dtype"]))
        out += [(k, j) for j in range(-(-nb // C))]
    return out


def _chunk_bytes(table, C, k, j, arena, key):
    e = table[k]
    nb = int(e["numel"]) * _esize(int(e["dtype"]))
    o = int(e[key]) + j * C
    return o, min(C, nb - j * C)


def _delta_offsets(table, C, ids, seg=SEGMENT):
    """Payload offset of each listed chunk (None if derived) and the payload
    size: a chunk right after the previous sent chunk of its entry follows it,
    any other starts at the next segment boundary."""
    cmap = _chunk_map(table, C)
    offs, end, prev = [], 0, None
    for c in ids:
        k, j = cmap[c]
        if int(table[k]["derive_from"]) >= 0:
            offs.append(None)
            continue
        _, ln = _chunk_bytes(table, C, k, j, None, "src_offset")
        offs.append(end if prev == (k, j - 1) else _up(end, seg))
        end = offs[-1] + ln
        prev = (k, j)
    return offs, _up(end, 16)


def pack_chunks(table, C, src: bytes, ids, seg=SEGMENT):
    cmap = _chunk_map(table, C)
    offs, size = _delta_offsets(table, C, ids, seg)
    payload = bytearray(size)
    sums = []
    for c, off in zip(ids, offs):
        k, j = cmap[c]
        o, ln = _chunk_bytes(table, C, k, j, src, "src_offset")
        if off is not None:
            payload[off:off + ln] = src[o:o + ln]
        sums.append(frsum(src[o:o + ln]))
    return bytes(payload), sums


def unpack_chunks(table, C, payload: bytes, sums, ids, dst: bytearray, seg=SEGMENT):
    cmap = _chunk_map(table, C)
    offs, _ = _delta_offsets(table, C, ids, seg)
    for c, off in zip(ids, offs):
        k, j = cmap[c]
        if off is not None:
            o, ln = _chunk_bytes(table, C, k, j, dst, "dst_offset")
            dst[o:o + ln] = payload[off:off + ln]
    for c in ids:
        k, j = cmap[c]
        s = int(table[k]["derive_from"])
        if s >= 0:
            o, ln = _chunk_bytes(table, C, k, j, dst, "dst_offset")
            mo = int(table[s]["dst_offset"]) + 2 * j * C
            for q in range(ln // 2):
                u = int.from_bytes(dst[mo + 4 * q:mo + 4 * q + 4], "little")
                dst[o + 2 * q:o + 2 * q + 2] = rne_bf16(u).to_bytes(2, "little")
    bad = set()
    for i, c in enumerate(ids):
        k, j = cmap[c]
        o, ln = _chunk_bytes(table, C, k, j, dst, "dst_offset")
        if frsum(bytes(dst[o:o + ln])) != tuple(sums[i]):
            bad.add(i)
    return bad
