"""Planted mistakes in the oracle are caught by its pins (CPU only).

Each mutant is a fresh copy of the Python oracle (``oracle/mini.py``) with
one plausible mistake planted in it: a dropped or shifted term, a wrong
index, a byte order, a modulus, a rounding rule, a layout constant, padding
left dirty, a delta layout or re-derivation order, the side a checksum reads or
the search that maps a chunk id to its tensor.  The pins that fix the oracle from outside it (hand-worked
values in tests/golden, closed forms, numpy's modular sums, torch's bf16
cast, exhaustive detection properties, independently built payloads, the
restore round trip) must accept the unmodified oracle and reject every
mutant: no plausible single mistake survives them.  The same is done for
the restatement of the controller's step-tag rules (oracle/steptag.py)
against the scenarios and the simulation of tests/test_steptag.py."""
import importlib.util
import os

import numpy as np
import pytest
import torch

from oracle import mini
from paper_2509_03047_amd import workloads as W

from tests.test_oracle_pins import _golden_frsum, _golden_rne

M64 = (1 << 64) - 1
MINI_PATH = mini.__file__


def _fresh_mini(tag):
    spec = importlib.util.spec_from_file_location(f"mini_mutant_{tag}", MINI_PATH)
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


# ---------------------------------------------------------------- pins

def frsum_pins(f, golden_dir):
    """Names of the FRSUM pins that `f` (bytes -> (sum, wsum)) fails."""
    failed = []
    if any(f(d) != (s, ws) for d, s, ws in _golden_frsum(golden_dir) if len(d) <= 65536):
        failed.append("golden")
    rng = np.random.default_rng(11)
    for n_words in (1, 3, 64, 1000):
        w = rng.integers(0, 1 << 32, size=n_words, dtype=np.uint64)
        with np.errstate(over="ignore"):
            s = int(np.sum(w, dtype=np.uint64))
            ws = int(np.sum(w * np.arange(1, n_words + 1, dtype=np.uint64), dtype=np.uint64))
        if f(w.astype("<u4").tobytes()) != (s, ws):
            failed.append("numpy")
            break
    n = 131072  # wsum of all-ones words wraps past 2^64 here
    if f(b"\xff" * (4 * n)) != ((n * 0xFFFFFFFF) & M64, (0xFFFFFFFF * n * (n + 1) // 2) & M64):
        failed.append("closed form")
    x = rng.integers(0, 256, size=200, dtype=np.uint8).tobytes()
    s0, ws0 = f(x)
    if f(bytes(20) + x) != (s0, (ws0 + 5 * s0) & M64):
        failed.append("shift law")
    if f(x[:198]) != f(x[:198] + b"\0\0") or f(b"\x80\x3f") != (16256, 16256):
        failed.append("bf16 tail")
    base = rng.integers(0, 256, size=16, dtype=np.uint8)
    ref = f(base.tobytes())
    for a in range(128):
        va = base.copy()
        va[a // 8] ^= np.uint8(1 << (a % 8))
        if f(va.tobytes())[0] == ref[0]:
            failed.append("single flips")
            break
        if any(f(_flip(va, b).tobytes()) == ref for b in range(a + 1, 128)):
            failed.append("double flips")
            break
    return failed


def _flip(v, bit):
    v = v.copy()
    v[bit // 8] ^= np.uint8(1 << (bit % 8))
    return v


def rne_pins(r, golden_dir):
    """Names of the rounding pins that `r` (fp32 bits -> bf16 bits) fails."""
    failed = []
    if any(r(u) != h for u, h in _golden_rne(golden_dir)):
        failed.append("golden")
    rng = np.random.default_rng(18)
    u = rng.integers(0, 1 << 32, size=4000, dtype=np.uint64).astype(np.uint32)
    # ties, denormals and values near overflow are rare among random
    # patterns: add them
    ties = (rng.integers(0, 1 << 16, size=500, dtype=np.uint64).astype(np.uint32) << np.uint32(16)) | np.uint32(0x8000)
    den = rng.integers(0, 1 << 23, size=500, dtype=np.uint64).astype(np.uint32)
    big = rng.integers(0x7F7F0000, 0x7F800000, size=500, dtype=np.uint64).astype(np.uint32)  # near overflow
    u = np.concatenate([u, ties, den, den | np.uint32(0x80000000), big, big | np.uint32(0x80000000)])
    u = u[(u & np.uint32(0x7FFFFFFF)) <= np.uint32(0x7F800000)]  # non-NaN
    ref = torch.from_numpy(u.view(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    if any(r(int(a)) != int(b) for a, b in zip(u, ref)):
        failed.append("torch cast")
    nan = [0x7F800001, 0xFF800001, 0x7FC00000, 0x7FFFFFFF, 0xFFA00000]
    if any(r(x) != ((x >> 16) | 0x40) for x in nan):
        failed.append("NaN reading")
    return failed


def layout_pins(m):
    """Names of the plan / pack / unpack pins that module `m` fails."""
    failed = []
    w = W.make_workload(0)  # table only: its closed forms need no state
    _, base, _, pb = m.plan(w.table, w.chunk_bytes)
    if pb != 12 * w.n_params or base[-1] != 804:
        failed.append("toy closed form")
    # 4 KiB segments: 14 gaps of 3 KiB after the 1 KiB norm arrays
    _, base, _, pb = m.plan(w.table, w.chunk_bytes, 4096)
    if pb != 12 * w.n_params + (5 * 3 - 1) * 3072 or base[-1] != 804:
        failed.append("toy closed form, 4 KiB segments")
    rng = np.random.default_rng(21)
    for seg in (16, 256, 4096):
        for _ in range(20):
            t, sb, db = W.random_tiny_table(rng)
            src = W.random_tiny_state(t, sb, rng).tobytes()
            payload, _ = m.pack(t, 64, src, seg)
            exp = bytearray()
            for e in t:
                if int(e["derive_from"]) >= 0:
                    continue
                o, n = int(e["src_offset"]), int(e["numel"]) * W.ESIZE[int(e["dtype"])]
                if n:
                    exp += bytes(-len(exp) % seg)
                    exp += src[o:o + n]
            exp += bytes(-len(exp) % 16)
            if bytes(payload) != bytes(exp):
                failed.append("concatenation")
                break
        if "concatenation" in failed:
            break
    t, nb = W.state_table([("a", 40), ("b", 3), ("c", 17)])
    src = W.random_tiny_state(t, nb, np.random.default_rng(23)).tobytes()
    payload, sums = m.pack(t, 32, src)
    dst = bytearray(nb)
    bad = m.unpack(t, 32, payload, sums, dst)
    if bad or bytes(dst) != src:
        failed.append("round trip")
    return failed


# ------------------------------------------------------------- mutants

def _frsum_with(word, weight, mask_s=M64, mask_ws=M64, tail=True, swap=False):
    def f(b):
        s = ws = 0
        step = 4
        n = len(b) if tail else len(b) - len(b) % 4
        for i in range(0, n, step):
            w = word(b[i:i + 4].ljust(4, b"\0"))
            s += w
            ws += weight(i) * w
        out = (s & mask_s, ws & mask_ws)
        return out[::-1] if swap else out
    return f


LE = lambda c: int.from_bytes(c, "little")  # noqa: E731
FRSUM_MUTANTS = {
    "weight is the 0-based index": _frsum_with(LE, lambda i: i // 4),
    "weight is the byte offset + 1": _frsum_with(LE, lambda i: i + 1),
    "big-endian words": _frsum_with(lambda c: int.from_bytes(c, "big"), lambda i: i // 4 + 1),
    "sum kept mod 2^32": _frsum_with(LE, lambda i: i // 4 + 1, mask_s=0xFFFFFFFF),
    "no wrap mod 2^64": _frsum_with(LE, lambda i: i // 4 + 1, mask_s=-1, mask_ws=-1),
    "short last word dropped": _frsum_with(LE, lambda i: i // 4 + 1, tail=False),
    "outputs swapped": _frsum_with(LE, lambda i: i // 4 + 1, swap=True),
    "16-bit words": lambda b: _frsum16(b),
}


def _frsum16(b):
    s = ws = 0
    for i in range(0, len(b), 2):
        w = int.from_bytes(b[i:i + 2].ljust(2, b"\0"), "little")
        s += w
        ws += (i // 2 + 1) * w
    return s & M64, ws & M64


def _nan_rule(u, h):
    return ((u >> 16) | 0x40) if (u & 0x7FFFFFFF) > 0x7F800000 else h


RNE_MUTANTS = {
    "truncation": lambda u: _nan_rule(u, u >> 16),
    "ties away from zero": lambda u: _nan_rule(u, (u + 0x8000) >> 16),
    "ties to odd": lambda u: _nan_rule(u, (u + 0x7FFF + (1 - ((u >> 16) & 1))) >> 16),
    "denormals flushed": lambda u: _nan_rule(
        u, (u >> 16) & 0x8000 if (u & 0x7F800000) == 0 else (u + 0x7FFF + ((u >> 16) & 1)) >> 16),
    "overflow saturates": lambda u: _nan_rule(u, min((u + 0x7FFF + ((u >> 16) & 1)) >> 16, 0x7F7F | (u >> 16 & 0x8000))
                                              if (u & 0x7FFFFFFF) < 0x7F800000 else u >> 16),
    "canonical NaN": lambda u: 0x7FC0 if (u & 0x7FFFFFFF) > 0x7F800000 else (u + 0x7FFF + ((u >> 16) & 1)) >> 16,
    "NaN not quieted": lambda u: (u >> 16) if (u & 0x7FFFFFFF) > 0x7F800000 else (u + 0x7FFF + ((u >> 16) & 1)) >> 16,
}


def _mutant_segment_fixed(a):
    def mutate(m):
        orig = m.plan
        m.plan = lambda table, C, seg=16: orig(table, C, a)
    return mutate


def _mutant_floor_chunks(m):
    orig = m.plan

    def plan(table, C, seg=16):
        nch, base, pay, pb = orig(table, C, seg)
        nch = [int(e["numel"]) * m._esize(int(e["dtype"])) // C for e in table]
        base = [0]
        for x in nch:
            base.append(base[-1] + x)
        return nch, base, pay, pb
    m.plan = plan


def _mutant_derived_sent(m):
    def plan(table, C, seg=16):
        nch, base, pay = [], [0], []
        end = 0
        for e in table:
            nb = int(e["numel"]) * m._esize(int(e["dtype"]))
            nch.append(-(-nb // C))
            base.append(base[-1] + nch[-1])
            pay.append(m._up(end, seg) if nb else m._up(end, 16))
            end = pay[-1] + nb if nb else end
        return nch, base, pay, m._up(end, 16)
    m.plan = plan


def _mutant_dirty_padding(m):
    orig = m.pack

    def pack(table, C, src, seg=16):
        payload, sums = orig(table, C, src, seg)
        p = bytearray(payload)
        _, _, pay, _ = m.plan(table, C, seg)
        used = bytearray(len(p))
        for k, e in enumerate(table):
            if pay[k] is not None:
                nb = int(e["numel"]) * m._esize(int(e["dtype"]))
                used[pay[k]:pay[k] + nb] = b"\1" * nb
        for i in range(len(p)):
            if not used[i]:
                p[i] = 0xFF
        return bytes(p), sums
    m.pack = pack


def _mutant_unrounded_end(m):
    orig = m.plan

    def plan(table, C, seg=16):
        nch, base, pay, pb = orig(table, C, seg)
        end = max([p + int(e["numel"]) * m._esize(int(e["dtype"]))
                   for p, e in zip(pay, table) if p is not None] + [0])
        return nch, base, pay, end
    m.plan = plan


def _mutant_truncating_rederive(m):
    m.rne_bf16 = lambda u: u >> 16


LAYOUT_MUTANTS = {
    "segments always on 4 KiB boundaries": _mutant_segment_fixed(4096),
    "segment alignment ignored (always 16)": _mutant_segment_fixed(16),
    "chunk count rounded down": _mutant_floor_chunks,
    "derived entries sent": _mutant_derived_sent,
    "padding not zeroed": _mutant_dirty_padding,
    "payload end not rounded to 16": _mutant_unrounded_end,
    "parameters re-derived by truncation": _mutant_truncating_rederive,
}


# --------------------------------------------------------------- tests

def test_pins_accept_the_oracle(golden_dir):
    assert frsum_pins(mini.frsum, golden_dir) == []
    assert rne_pins(mini.rne_bf16, golden_dir) == []
    assert layout_pins(_fresh_mini("clean")) == []


@pytest.mark.parametrize("name", sorted(FRSUM_MUTANTS))
def test_frsum_mutant_is_caught(name, golden_dir):
    assert frsum_pins(FRSUM_MUTANTS[name], golden_dir), name


@pytest.mark.parametrize("name", sorted(RNE_MUTANTS))
def test_rne_mutant_is_caught(name, golden_dir):
    assert rne_pins(RNE_MUTANTS[name], golden_dir), name


@pytest.mark.parametrize("name", sorted(LAYOUT_MUTANTS))
def test_layout_mutant_is_caught(name):
    m = _fresh_mini(name.replace(" ", "_"))
    LAYOUT_MUTANTS[name](m)
    assert layout_pins(m), name


# ------------------------------------------------------ checksum paths

def checksum_pins(m):
    """Names of the checksum-path pins (one replica's checksum, the replica
    compare's sums, the checksum of a chunk list) that module `m` fails: the
    hand-worked scattered table, and the location of single flipped bits on
    random scattered tables with empty entries, walked in the test."""
    from tests.test_oracle_checksum import (_chunk_of_byte, _edge_ids, load_checksum_golden,
                                            with_empty_entries)

    failed = []
    t, C, a, sums, ids, list_sums, b, diff, sums_b = load_checksum_golden()
    ab, bb = a.tobytes(), b.tobytes()
    if m.checksum(t, C, ab) != sums:
        failed.append("worked checksum")
    if m.verify_with_sums(t, C, ab, bb) != (diff, sums, sums_b):
        failed.append("worked compare sums")
    if m.checksum_chunks(t, C, ab, ids) != list_sums:
        failed.append("worked chunk list")
    rng = np.random.default_rng(91)
    for _ in range(40):
        t0, sb, db = W.random_tiny_table(rng, max_entries=5, max_numel=120)
        t = with_empty_entries(t0, sb, db, rng)
        C = int(rng.choice([16, 32, 64]))
        x = W.random_tiny_state(t, sb, rng)
        ref = m.checksum(t, C, x.tobytes())
        if sb:
            p = int(rng.integers(0, sb))
            y = x.copy()
            y[p] ^= np.uint8(1)
            got = m.checksum(t, C, y.tobytes())
            c = _chunk_of_byte(t, C, p)
            changed = {i for i, (u, v) in enumerate(zip(ref, got)) if u != v}
            if changed != (set() if c is None else {c}):
                failed.append("flip location")
                break
        edge = _edge_ids(t, C)
        if m.checksum_chunks(t, C, x.tobytes(), edge) != [ref[i] for i in edge]:
            failed.append("chunk list next to empty entries")
            break
    return failed


def _mutant_sums_at_dst(m):
    m.checksum = lambda table, C, arena: [m.frsum(b) for _, b in m._chunks(table, C, arena, "dst_offset")]


def _mutant_search_off_by_one(m):
    def entry_of(base, c):
        lo, hi = 0, len(base) - 1
        while hi - lo > 1:
            mid = (lo + hi) // 2
            if base[mid] < c:
                lo = mid
            else:
                hi = mid
        return lo
    m._entry_of = entry_of


CHECKSUM_MUTANTS = {
    "sums read at dst offsets": _mutant_sums_at_dst,
    "chunk search off by one": _mutant_search_off_by_one,
}


def test_checksum_pins_accept_the_oracle():
    assert checksum_pins(_fresh_mini("checksum_clean")) == []


@pytest.mark.parametrize("name", sorted(CHECKSUM_MUTANTS))
def test_checksum_mutant_is_caught(name):
    m = _fresh_mini(name.replace(" ", "_"))
    CHECKSUM_MUTANTS[name](m)
    assert checksum_pins(m), name


# ----------------------------------------------------------- delta repair

def delta_pins(m):
    """Names of the delta-repair pins that module `m` fails."""
    failed = []
    rng = np.random.default_rng(61)
    for it in range(60):
        t, sb, db = W.random_tiny_table(rng, max_numel=120)
        C = int(rng.choice([16, 32, 64]))
        seg = (16, 64, 4096)[it % 3]
        src = W.random_tiny_state(t, sb, rng).tobytes()
        n = len(m._chunk_map(t, C))
        fp, fs = m.pack(t, C, src, seg)
        dp, ds = m.pack_chunks(t, C, src, list(range(n)), seg)
        if dp != fp or [tuple(x) for x in ds] != [tuple(x) for x in fs]:
            failed.append("full list is the full pack")
            break
    # a list with gaps, worked by hand (16-byte chunks, 64-byte segments):
    # chunk 0 at 0; chunks 2-3 (a run) at 64; chunk 9 at 128; chunk 10 (the
    # next entry's first) at 192; payload 208 bytes
    t = np.array([(0, 0, 40, W.F32, -1), (160, 160, 8, W.F32, -1)], dtype=W.TABLE_DTYPE)
    src = bytes(range(192))
    pay, _ = m.pack_chunks(t, 16, src, [0, 2, 3, 9, 10], 64)
    exp = (src[0:16] + bytes(48) + src[32:64] + bytes(32) + src[144:160] + bytes(48)
           + src[160:176])
    if pay != exp:
        failed.append("runs start segments")
    # repair of a replica whose master, its bf16 image and a moment diverged
    t, nb = W.state_table([("a", 40), ("b", 3), ("c", 17)])
    donor = W.random_tiny_state(t, nb, np.random.default_rng(23)).tobytes()
    recv = bytearray(donor)
    m0, p0, v0 = int(t[1]["src_offset"]), int(t[0]["src_offset"]), int(t[3]["src_offset"])
    for o, x in ((m0 + 67, 0x40), (p0 + 33, 0x01), (v0 + 5, 0x80), (m0 + 3, 0x02)):
        recv[o] ^= x
    for C in (16, 32, 64):
        r = bytearray(recv)
        ids = sorted(m.verify(t, C, donor, bytes(r)))
        pay, sums = m.pack_chunks(t, C, donor, ids)
        bad = m.unpack_chunks(t, C, pay, sums, ids, r)
        if bad or bytes(r) != donor:
            failed.append("repair restores the donor")
            break
    return failed


def _delta_offsets_with(m, rule):
    def offsets(table, C, ids, seg=16):
        cmap = m._chunk_map(table, C)
        offs, end, prev = [], 0, None
        for c in ids:
            k, j = cmap[c]
            if int(table[k]["derive_from"]) >= 0:
                offs.append(None)
                continue
            _, ln = m._chunk_bytes(table, C, k, j, None, "src_offset")
            offs.append(rule(end, prev == (k, j - 1), seg))
            end = offs[-1] + ln
            prev = (k, j)
        return offs, m._up(end, 16)
    m._delta_offsets = offsets


def _unpack_chunks_with(m, derive_first=False, master_index=2):
    def unpack_chunks(table, C, payload, sums, ids, dst, seg=16):
        cmap = m._chunk_map(table, C)
        offs, _ = m._delta_offsets(table, C, ids, seg)

        def sent():
            for c, off in zip(ids, offs):
                k, j = cmap[c]
                if off is not None:
                    o, ln = m._chunk_bytes(table, C, k, j, dst, "dst_offset")
                    dst[o:o + ln] = payload[off:off + ln]

        def derived():
            for c in ids:
                k, j = cmap[c]
                s = int(table[k]["derive_from"])
                if s >= 0:
                    o, ln = m._chunk_bytes(table, C, k, j, dst, "dst_offset")
                    mo = int(table[s]["dst_offset"]) + master_index * j * C
                    for q in range(ln // 2):
                        u = int.from_bytes(dst[mo + 4 * q:mo + 4 * q + 4], "little")
                        dst[o + 2 * q:o + 2 * q + 2] = m.rne_bf16(u).to_bytes(2, "little")
        for step in ((derived, sent) if derive_first else (sent, derived)):
            step()
        bad = set()
        for i, c in enumerate(ids):
            k, j = cmap[c]
            o, ln = m._chunk_bytes(table, C, k, j, dst, "dst_offset")
            if m.frsum(bytes(dst[o:o + ln])) != tuple(sums[i]):
                bad.add(i)
        return bad
    m.unpack_chunks = unpack_chunks


DELTA_MUTANTS = {
    "every chunk on a new segment": lambda m: _delta_offsets_with(
        m, lambda end, cont, seg: m._up(end, seg)),
    "no segment boundaries": lambda m: _delta_offsets_with(m, lambda end, cont, seg: end),
    "segments on 16-byte boundaries whatever the alignment": lambda m: _delta_offsets_with(
        m, lambda end, cont, seg: end if cont else m._up(end, 16)),
    "parameters re-derived before the masters land": lambda m: _unpack_chunks_with(m, derive_first=True),
    "parameter chunk j read from master chunk j": lambda m: _unpack_chunks_with(m, master_index=1),
}


def test_delta_pins_accept_the_oracle():
    assert delta_pins(_fresh_mini("delta_clean")) == []


@pytest.mark.parametrize("name", sorted(DELTA_MUTANTS))
def test_delta_mutant_is_caught(name):
    m = _fresh_mini("delta_" + name.replace(" ", "_"))
    DELTA_MUTANTS[name](m)
    assert delta_pins(m), name


# ------------------------------------------------------- step-tag tracker

from oracle.steptag import Cluster  # noqa: E402

from tests import test_steptag as S  # noqa: E402


class _NoFreshness(Cluster):
    """Trusts tags reported before the failure was detected."""

    def decide(self, now):
        saved = dict(self.seen)
        self.seen = {r: float("inf") for r in saved}
        try:
            return Cluster.decide(self, now)
        finally:
            self.seen = saved


class _OptimizerTagIsAStep(Cluster):
    """Does not wait for ranks inside their optimizer step (tag -1)."""

    def decide(self, now):
        saved = dict(self.tag)
        self.tag = {r: (10 ** 9 if v == -1 else v) for r, v in saved.items()}
        try:
            a, s = Cluster.decide(self, now)
            return (a, -1 if s == 10 ** 9 else s)
        finally:
            self.tag = saved


class _FallbackOnAnyLoss(Cluster):
    """Falls back to a checkpoint as soon as a group lost any member, not
    only when it lost every member."""

    def decide(self, now):
        if self.failed(now):
            return "checkpoint_fallback", -1
        return Cluster.decide(self, now)


class _NoTimeout(Cluster):
    """Detects only reported failures (a silent rank is never failed)."""

    def failed(self, now):
        return [r for r in range(self.n_ranks) if r in self.reported]


class _ResumeAfterTag(Cluster):
    """Resumes one step after the agreed tag."""

    def decide(self, now):
        a, s = Cluster.decide(self, now)
        return (a, s + 1 if a == "stop_and_restore" else s)


STEPTAG_MUTANTS = {
    "stale tags trusted": _NoFreshness,
    "optimizer-step tag not waited for": _OptimizerTagIsAStep,
    "checkpoint when any replica is lost": _FallbackOnAnyLoss,
    "silent ranks never time out": _NoTimeout,
    "resume one step late": _ResumeAfterTag,
}


def _steptag_pins_failed(cluster_cls):
    class Make(S.OracleTracker):
        cluster = cluster_cls
    failed = []
    for name in dir(S):
        fn = getattr(S, name)
        if name.startswith("test_") and callable(fn) and fn.__code__.co_varnames[:1] == ("make",):
            try:
                fn(Make)
            except AssertionError:
                failed.append(name)
    for seed in range(40):
        try:
            S.check_simulation(seed, Make)
        except AssertionError:
            failed.append(f"simulation {seed}")
    return failed


def test_steptag_pins_accept_the_oracle():
    assert _steptag_pins_failed(Cluster) == []


@pytest.mark.parametrize("name", sorted(STEPTAG_MUTANTS))
def test_steptag_mutant_is_caught(name):
    assert _steptag_pins_failed(STEPTAG_MUTANTS[name]), name


# ------------------------------------------------------- restore planner

from oracle import planner as _planner  # noqa: E402


def _fresh_planner(tag):
    spec = importlib.util.spec_from_file_location(f"planner_mutant_{tag}", _planner.__file__)
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


PLANNER_LAYOUTS = [(1, 1, 4, 1), (2, 1, 4, 1), (2, 2, 4, 2), (1, 2, 8, 4), (2, 2, 4, 4), (4, 1, 2, 2),
                   (2, 3, 6, 2)]


def planner_pins(P):
    """Names of the planner pins that module P fails.  Replica classes must
    partition the ranks into groups of dp / shard ranks holding identical
    state (equal tensor-parallel index, pipeline stage and shard); a donor
    must be a live member of the failed rank's class, -1 when none is left,
    and donors spread evenly over a class's live members."""
    failed = []
    rng = np.random.default_rng(5)
    for tp, pp, dp, shard in PLANNER_LAYOUTS:
        world = tp * pp * dp
        state = {r: (lambda c: (c[0], c[1], c[3]))(_planner.coords(tp, pp, dp, shard, r)) for r in range(world)}
        for r in range(world):
            reps = P.replicas(tp, pp, dp, shard, r)
            if (r not in reps or len(set(reps)) != dp // shard
                    or any(not 0 <= x < world or state[x] != state[r] for x in reps)):
                failed.append("replica classes")
                return failed
        for _ in range(20):
            dead = set(int(x) for x in rng.choice(world, size=int(rng.integers(0, world + 1)), replace=False))
            d = P.donors(tp, pp, dp, shard, dead)
            loads = {}
            for r in range(world):
                live = [x for x in range(world) if state[x] == state[r] and x not in dead]
                if r not in dead or not live:
                    if d[r] != -1:
                        failed.append("donor for a live or unservable rank")
                        return failed
                    continue
                if d[r] not in live:
                    failed.append("donor is a live replica")
                    return failed
                loads.setdefault(state[r], []).append(d[r])
            for cls, used in loads.items():
                live = [x for x in range(world) if state[x] == cls and x not in dead]
                counts = [used.count(x) for x in live]
                if max(counts) - min(counts) > 1:
                    failed.append("even spread")
                    return failed
    return failed


def _pl_replicas_no_stage(P):
    def replicas(tp, pp, dp, shard, rank):
        t, p, d, s, q = P.coords(tp, pp, dp, shard, rank)
        return [t + tp * (s + shard * qq) for qq in range(dp // shard)]
    P.replicas = replicas


def _pl_replicas_over_shards(P):
    def replicas(tp, pp, dp, shard, rank):
        t, p, d, s, q = P.coords(tp, pp, dp, shard, rank)
        return [t + tp * (ss + shard * q + dp * p) for ss in range(shard)] if shard > 1 else \
            [t + tp * (s + shard * qq + dp * p) for qq in range(dp)]
    P.replicas = replicas


def _pl_first_live_donor(P):
    def donors(tp, pp, dp, shard, failed):
        out = [-1] * (tp * pp * dp)
        for r in failed:
            live = [x for x in sorted(P.replicas(tp, pp, dp, shard, r)) if x not in failed]
            if live:
                out[r] = live[0]
        return out
    P.donors = donors


def _pl_failed_donor(P):
    def donors(tp, pp, dp, shard, failed):
        out = [-1] * (tp * pp * dp)
        served = {}
        for r in sorted(failed):
            reps = sorted(P.replicas(tp, pp, dp, shard, r))
            if any(x not in failed for x in reps):
                k = served.get(tuple(reps), 0)
                out[r] = reps[k % len(reps)]
                served[tuple(reps)] = k + 1
        return out
    P.donors = donors


PLANNER_MUTANTS = {
    "replicas ignore the pipeline stage": _pl_replicas_no_stage,
    "replicas run over the shard index": _pl_replicas_over_shards,
    "always the first live replica": _pl_first_live_donor,
    "failed ranks may donate": _pl_failed_donor,
}


def test_planner_pins_accept_the_oracle():
    assert planner_pins(_fresh_planner("clean")) == []


@pytest.mark.parametrize("name", sorted(PLANNER_MUTANTS))
def test_planner_mutant_is_caught(name):
    P = _fresh_planner(name.replace(" ", "_"))
    PLANNER_MUTANTS[name](P)
    assert planner_pins(P), name


# ------------------------------------------ consistency from sums alone

COMPARE_MUTANTS = {
    "sum field only": lambda sa, sb: {c for c, (x, y) in enumerate(zip(sa, sb)) if x[0] != y[0]},
    "wsum field only": lambda sa, sb: {c for c, (x, y) in enumerate(zip(sa, sb)) if x[1] != y[1]},
    "chunk ids off by one": lambda sa, sb: {c + 1 for c, (x, y) in enumerate(zip(sa, sb)) if x != y},
    "last chunk dropped": lambda sa, sb: {c for c, (x, y) in enumerate(zip(sa[:-1], sb[:-1])) if x != y},
}


def test_compare_pins_accept_the_oracle():
    from tests.test_oracle_checksum import compare_pins

    assert compare_pins(_fresh_mini("compare_clean").compare_sums, mini.checksum) == []


@pytest.mark.parametrize("name", sorted(COMPARE_MUTANTS))
def test_compare_mutant_is_caught(name):
    from tests.test_oracle_checksum import compare_pins

    assert compare_pins(COMPARE_MUTANTS[name], mini.checksum), name
