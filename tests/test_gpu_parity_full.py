"""GPU parity at full workload sizes, in the launch configuration the benchmark
times (default plan, one workgroup per unit).

* Llama-3-8B TP=8 rank share (14.06 GB state): the whole oracle runs on the
  host; payload, sums, receiver arena and result sets are compared bit for bit,
  at 64 KiB chunks and at 1 KiB chunks (the tiles chosen by chunk size).
* 20,000-entry descriptor stress (7.6 GB): whole oracle, scattered layouts,
  canaries in every receiver gap, at 16-byte and 4 KiB payload segments;
  its replica compare (line-aligned, since its tensors start inside cache
  lines) with flips at chunk and line edges.
* Llama-3-70B TP=8 x PP=4 first-stage share (31.8 GB): the whole oracle on
  the host (payload, sums and receiver arena compared slice by slice), plus
  sampled chunks, a located wire flip and properties that hold at any size
  (exact round trip, nothing flagged, checksum == pack sums, replica compare
  empty); a replica with 4,096 flips: compare set, both arenas' sums and the
  checksum against the whole oracle.
* One tensor of 1.2 G parameters (16.8 GB state): offsets past 2^32 bytes
  inside one entry, whole oracle and a wire flip 4.5 GB into the master.
* Replica compare on two copies of the 8B share with k in {0, 1, 64, 4096}
  distinct random bit flips: the flagged set equals the closed form
  {chunk of each flipped byte} and the oracle's set; the 4,096-flip replica
  repaired by a delta (payload and sums against the oracle).
"""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from tests.gpu_util import Restore, log, sums_host, to_host  # noqa: E402


@pytest.fixture(scope="module")
def llama8b():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(1)
    import time

    t0 = time.perf_counter()
    src = W.fill_state(w)
    log(f"generated {w.name} ({w.state_bytes} B) in {time.perf_counter() - t0:.1f} s")
    return w, src


def _upload(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(a).to("cuda")


def _flip_on_device(t: torch.Tensor, bit_positions: np.ndarray):
    """XOR distinct bit positions into a device byte tensor (bytes may repeat)."""
    if bit_positions.size == 0:
        return
    by = (bit_positions // 8).astype(np.int64)
    masks = (np.uint8(1) << (bit_positions % 8).astype(np.uint8)).astype(np.uint8)
    order = np.argsort(by, kind="stable")
    by, masks = by[order], masks[order]
    uniq, start = np.unique(by, return_index=True)
    comb = np.bitwise_or.reduceat(masks, start)
    idx = torch.from_numpy(uniq).to("cuda")
    m = torch.from_numpy(comb).to("cuda")
    t[idx] = t[idx] ^ m


def _expected_chunks(w, plan_base, bit_positions):
    starts = w.table["src_offset"].astype(np.int64)
    out = set()
    for p in bit_positions:
        byte = int(p) // 8
        e = int(np.searchsorted(starts, byte, side="right") - 1)
        out.add(int(plan_base[e]) + (byte - int(starts[e])) // w.chunk_bytes)
    return out


@pytest.mark.timeout(900)
def test_llama8b_tp8_full_parity(llama8b):
    w, src_np = llama8b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    r.verify(src, r.dst)
    r.checksum(r.dst)
    torch.cuda.synchronize()
    log("gpu ops done")
    pay, sums = cpu.pack(t, C, src_np)
    log("oracle pack done")
    nc = r.n_chunks
    assert nc == 214_684 and pay.size == 12_048_187_392
    assert np.array_equal(sums_host(r.sums, nc), sums)
    g_pay = to_host(r.payload)
    assert np.array_equal(g_pay[: pay.size], pay)
    del g_pay
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    log("oracle unpack done")
    assert nbad == 0 and int(r.n_bad.item()) == 0 and r.bad_set() == set()
    assert np.array_equal(to_host(r.dst), dst)
    assert int(r.n_diff.item()) == 0 and r.diff_set() == set()
    assert np.array_equal(sums_host(r.csum, nc), sums)


@pytest.mark.timeout(900)
def test_llama8b_1kib_chunks_full_parity(llama8b, monkeypatch):
    """The 8B share in 1 KiB chunks (13.7 million chunks) with the tiles chosen
    by chunk size (unpack and compare 64 x 1, checksum 64 x 4): whole
    oracle for pack, unpack, compare and checksum."""
    for k in [k for k in os.environ if k.startswith("FLASHRESTORE_TILE")]:
        monkeypatch.delenv(k)
    w, src_np = llama8b
    t, C = w.table, 1024
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5)
    info = r.plan.info
    assert (info["tile_pack"], info["tile_unpack"], info["tile_verify"], info["tile_checksum"]) == (4, 7, 7, 4)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    r.verify(src, r.dst)
    r.checksum(r.dst)
    torch.cuda.synchronize()
    log("gpu ops done")
    pay, sums = cpu.pack(t, C, src_np)
    nc = r.n_chunks
    assert nc > 13_000_000
    assert np.array_equal(sums_host(r.sums, nc), sums)
    assert np.array_equal(to_host(r.payload)[: pay.size], pay)
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    log("oracle done")
    assert nbad == 0 and int(r.n_bad.item()) == 0 and r.bad_set() == set()
    assert np.array_equal(to_host(r.dst), dst)
    assert int(r.n_diff.item()) == 0 and r.diff_set() == set()
    assert np.array_equal(sums_host(r.csum, nc), sums)


@pytest.fixture
def over_4gib():
    """A table whose middle tensor has 1.2 G parameters: its fp32 master, m
    and v are 4.8 GB entries each, past 2^32 bytes inside one entry."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tensors = [("head", 3_001), ("huge", 1_200_000_000), ("tail", 70_001)]
    table, nb = W.state_table(tensors)
    w = W.Workload("one-tensor-over-4GiB", table, 1 << 20, nb, nb, tensors, 7)
    log(f"generating {w.name} ({w.state_bytes} B)")
    return w, W.fill_state(w)


@pytest.mark.timeout(900)
def test_tensor_over_4gib_full_parity(over_4gib):
    """Offsets past 2^32 bytes inside one entry: the master, m and v of one
    tensor are 4.8 GB each, its bf16 image (2.4 GB) is re-derived from master
    bytes read up to 4.8 GB into the entry, and the last tensor starts past
    16 GB.  Whole oracle: payload, sums, receiver arena (canaries in the
    padding), flags, compare and checksum; then a wire flip 4.5 GB into the
    master's payload is flagged as the oracle flags it."""
    w, src_np = over_4gib
    t, C = w.table, w.chunk_bytes
    assert int(t["numel"][5]) * 4 > (1 << 32) and int(t["src_offset"][8]) > 16 * 10**9
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    r.verify(src, r.dst)
    r.checksum(r.dst)
    torch.cuda.synchronize()
    log("gpu ops done")
    pay, sums = cpu.pack(t, C, src_np)
    log("oracle pack done")
    nc = r.n_chunks
    assert np.array_equal(sums_host(r.sums, nc), sums)
    g_pay = to_host(r.payload)
    assert np.array_equal(g_pay[: pay.size], pay)
    del g_pay
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    log("oracle unpack done")
    assert nbad == 0 and int(r.n_bad.item()) == 0 and r.bad_set() == set()
    assert np.array_equal(to_host(r.dst), dst)
    assert int(r.n_diff.item()) == 0 and r.diff_set() == set()
    assert np.array_equal(sums_host(r.csum, nc), sums)
    # a wire flip 4.5 GB into the huge master's payload segment
    info, pay_of_entry, base = F.fr_layout_query(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    byte = int(pay_of_entry[5]) + 4_500_000_003
    pay[byte] ^= np.uint8(0x10)
    r.payload[byte] ^= 0x10
    r.dst.fill_(0xA5)
    r.unpack()
    dst.fill(0xA5)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    log("flipped unpack done")
    want = set(cpu.bitmap_to_set(bm, nc))
    assert int(base[5]) + 4_500_000_003 // C in want
    assert r.bad_set() == want and int(r.n_bad.item()) == nbad
    assert np.array_equal(to_host(r.dst), dst)


@pytest.mark.timeout(900)
def test_llama8b_replica_verify_flips(llama8b):
    w, a_np = llama8b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    a = _upload(a_np)
    b = a.clone()
    base = cpu.plan(t, C)[1]
    nc = r.n_chunks
    ref_sums = cpu.checksum(t, C, a_np)
    log("oracle checksum of A done")
    for k in (0, 1, 64, 4096):
        pos = W.flip_positions(a_np.size * 8, k, 4000 + k)
        exp = _expected_chunks(w, base, pos)
        _flip_on_device(b, pos)
        sa, sb = r.plan.empty_sums(), r.plan.empty_sums()
        r.verify(a, b, sa, sb)
        got = r.diff_set()
        assert got == exp, f"k={k}"
        assert int(r.n_diff.item()) == len(exp)
        # the oracle's exact compare on the same bytes
        b_np = a_np.copy()
        W.apply_flips(b_np, pos)
        vb, nd = cpu.verify(t, C, a_np, b_np)
        assert set(cpu.bitmap_to_set(vb, nc)) == exp and nd == len(exp)
        # sums of A equal the oracle's; sums of B differ exactly on the set
        g_sa, g_sb = sums_host(sa, nc), sums_host(sb, nc)
        assert np.array_equal(g_sa, ref_sums)
        ids = np.array(sorted(exp), dtype=np.uint64)
        if ids.size:
            assert np.array_equal(g_sb.reshape(-1, 2)[ids.astype(np.int64)].reshape(-1),
                                  cpu.checksum_chunks(t, C, b_np, ids))
        same = np.ones(nc, bool)
        same[ids.astype(np.int64)] = False
        assert np.array_equal(g_sb.reshape(-1, 2)[same], g_sa.reshape(-1, 2)[same])
        # a compare of sums alone would find the same set: no flipped chunk's
        # (sum, wsum) is unchanged
        if ids.size:
            ii = ids.astype(np.int64)
            moved = (g_sb.reshape(-1, 2)[ii] != g_sa.reshape(-1, 2)[ii]).any(axis=1)
            assert moved.all(), f"checksum collisions at k={k}: {ids[~moved].tolist()}"
        # ... and fr_compare_sums on the two sums arrays finds it, as the
        # oracle's compare of the same sums does
        cbm, cnd = r.plan.empty_bitmap(), r.plan.empty_counter()
        got_s = set(int(c) for c in r.plan.compare_sums(sa, sb, cbm, cnd, sync=True))
        obm, ond = cpu.compare_sums(ref_sums, cpu.checksum(t, C, b_np))
        assert got_s == exp == set(cpu.bitmap_to_set(obm, nc)) and int(cnd.item()) == ond == len(exp)
        del b_np
        _flip_on_device(b, pos)  # restore B
        log(f"replica verify k={k}: {len(exp)} chunks")
    r.verify(a, b)
    assert r.diff_set() == set()


@pytest.mark.timeout(900)
def test_descriptor_stress_full_parity():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(2)
    t, C = w.table, w.chunk_bytes
    src_np = W.fill_state(w)
    log(f"generated {w.name}: {len(t)} entries, {w.state_bytes} B")
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    r.checksum(src)
    torch.cuda.synchronize()
    pay, sums = cpu.pack(t, C, src_np)
    nc = r.n_chunks
    assert np.array_equal(sums_host(r.sums, nc), sums)
    assert np.array_equal(to_host(r.payload)[: pay.size], pay)
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    assert nbad == 0 and r.bad_set() == set() and int(r.n_bad.item()) == 0
    assert np.array_equal(to_host(r.dst), dst)
    assert np.array_equal(sums_host(r.csum, nc), sums)
    # a corrupted wire on this layout: three payload flips
    rng = np.random.default_rng(5)
    for _ in range(3):
        bit = int(rng.integers(0, pay.size * 8))
        pay[bit // 8] ^= np.uint8(1 << (bit % 8))
        r.payload[bit // 8] ^= 1 << (bit % 8)
    r.unpack()
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst)
    assert r.bad_set() == set(cpu.bitmap_to_set(bm, nc)) and int(r.n_bad.item()) == nbad


@pytest.mark.timeout(900)
def test_descriptor_stress_4kib_segments_full_parity():
    """The stress table with the 4 KiB payload-segment wire format (every
    segment starts on a 4 KiB boundary, gaps zero): pack walks plain slices,
    unpack walks receiver tiles; whole oracle at that alignment, and a
    corrupted wire."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(2)
    t, C = w.table, w.chunk_bytes
    src_np = W.fill_state(w)
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5, seg=4096)
    assert (r.plan.info["pack_walk"], r.plan.info["unpack_walk"]) == (0, 4)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    torch.cuda.synchronize()
    pay, sums = cpu.pack(t, C, src_np, 4096)
    nc = r.n_chunks
    assert np.array_equal(sums_host(r.sums, nc), sums)
    assert np.array_equal(to_host(r.payload)[: pay.size], pay)
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst, 4096)
    assert nbad == 0 and r.bad_set() == set() and int(r.n_bad.item()) == 0
    assert np.array_equal(to_host(r.dst), dst)
    rng = np.random.default_rng(6)
    for _ in range(3):
        bit = int(rng.integers(0, pay.size * 8))
        pay[bit // 8] ^= np.uint8(1 << (bit % 8))
        r.payload[bit // 8] ^= 1 << (bit % 8)
    r.unpack()
    dst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    bm, nbad = cpu.unpack(t, C, pay, sums, dst, 4096)
    assert r.bad_set() == set(cpu.bitmap_to_set(bm, nc)) and int(r.n_bad.item()) == nbad
    assert np.array_equal(to_host(r.dst), dst)


@pytest.mark.timeout(900)
def test_descriptor_stress_replica_compare():
    """The replica compare on the stress table, whose tensors start inside
    cache lines (the compare walks line-aligned there): bits flipped at chunk
    starts and ends, next to line boundaries and at random give the oracle's
    set and both arenas' sums, and the set is the closed form {chunk of each
    flipped byte inside a tensor}."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(2)
    t, C = w.table, w.chunk_bytes
    src_np = W.fill_state(w)
    rng = np.random.default_rng(11)
    nb = t["numel"].astype(np.int64) * np.where(t["dtype"] == W.F32, 4, 2)
    so = t["src_offset"].astype(np.int64)
    picks = []
    for e in rng.choice(len(t), size=200, replace=False):
        e = int(e)
        n = int(nb[e])
        j = int(rng.integers(0, -(-n // C)))
        lo, hi = j * C, min((j + 1) * C, n)
        line = (-(int(so[e]) + lo)) % 128  # first line boundary inside the chunk
        for off in (lo, lo + 1, lo + line, lo + line - 1, hi - 1, int(rng.integers(lo, hi))):
            if lo <= off < hi:
                picks.append(int(so[e]) + off)
    pos = np.unique(np.array(picks, np.int64)) * 8 + rng.integers(0, 8, size=len(set(picks)))
    b_np = src_np.copy()
    W.apply_flips(b_np, pos)
    a, b = _upload(src_np), _upload(b_np)
    plan = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes).plan
    diff, nd = plan.empty_bitmap(), plan.empty_counter()
    sa, sb = plan.empty_sums(), plan.empty_sums()
    got = plan.verify_replicas(a, b, diff, nd, sa, sb, sync=True)
    vbm, ond, osa, osb = cpu.verify(t, C, src_np, b_np, with_sums=True)
    nc = plan.n_chunks
    assert set(int(x) for x in got) == set(cpu.bitmap_to_set(vbm, nc)) and int(nd.item()) == ond
    assert np.array_equal(sums_host(sa, nc), osa) and np.array_equal(sums_host(sb, nc), osb)
    _, base, _, _ = cpu.plan(t, C)
    order = np.argsort(so, kind="stable")  # the table is shuffled over the arena
    exp = set()
    for byte in pos // 8:
        i = int(np.searchsorted(so[order], byte, side="right") - 1)
        e = int(order[i]) if i >= 0 else -1
        if e >= 0 and byte - so[e] < nb[e]:
            exp.add(int(base[e]) + int(byte - so[e]) // C)
    assert set(int(x) for x in got) == exp
    log(f"stress compare: {len(pos)} flips, {len(exp)} chunks flagged")


@pytest.fixture(scope="module")
def llama70b():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(3)
    src = W.fill_state(w)
    log(f"generated {w.name}: {w.state_bytes} B")
    return w, src


def _equal_in_slices(dev: torch.Tensor, host: np.ndarray, step: int = 1 << 30) -> bool:
    """Device bytes equal host bytes, copied back one slice at a time."""
    if dev.numel() < host.size:
        return False
    for a in range(0, host.size, step):
        b = min(a + step, host.size)
        if not np.array_equal(to_host(dev[a:b]), host[a:b]):
            log(f"mismatch in bytes [{a}, {b})")
            return False
    return True


@pytest.mark.timeout(900)
def test_llama70b_stage0_whole_oracle_parity(llama70b):
    w, src_np = llama70b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    r.pack(_upload(src_np))
    r.unpack()
    torch.cuda.synchronize()
    nc = r.n_chunks
    opay, osums = cpu.pack(t, C, src_np)
    log("oracle pack done")
    assert opay.size == r.plan.payload_bytes
    assert np.array_equal(sums_host(r.sums, nc), osums)
    assert _equal_in_slices(r.payload, opay)
    log("payload and sums equal the oracle's")
    odst = np.full(w.dst_arena_bytes, 0xA5, np.uint8)
    obm, onbad = cpu.unpack(t, C, opay, osums, odst)
    del opay
    log("oracle unpack done")
    assert onbad == 0 and int(r.n_bad.item()) == 0 and r.bad_set() == set()
    assert _equal_in_slices(r.dst, odst)
    log("receiver arena equals the oracle's")


@pytest.mark.timeout(900)
def test_llama70b_stage0_sampled_parity(llama70b):
    w, src_np = llama70b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    src = _upload(src_np)
    r.pack(src)
    r.unpack()
    r.verify(src, r.dst)
    r.checksum(r.dst)
    torch.cuda.synchronize()
    nc = r.n_chunks
    assert nc == 30_474
    # properties at full size
    assert int(r.n_bad.item()) == 0 and int(r.n_diff.item()) == 0
    assert torch.equal(r.dst, src)
    assert torch.equal(r.csum[:nc], r.sums[:nc])
    # sampled chunks against the oracle, one by one
    _, base, pay_off, pb = cpu.plan(t, C)
    assert pb == r.plan.payload_bytes == 27_249_082_368
    rng = np.random.default_rng(33)
    ids = np.unique(np.concatenate([rng.integers(0, nc, 512), [0, nc - 1]])).astype(np.uint64)
    exp = cpu.checksum_chunks(t, C, src_np, ids)
    assert np.array_equal(sums_host(r.sums, nc).reshape(-1, 2)[ids.astype(np.int64)].reshape(-1), exp)
    for c in ids[:64]:
        c = int(c)
        k = int(np.searchsorted(base, c, side="right") - 1)
        j = c - int(base[k])
        nb = int(t[k]["numel"]) * W.ESIZE[int(t[k]["dtype"])]
        ln = min(C, nb - j * C)
        so = int(t[k]["src_offset"]) + j * C
        if int(t[k]["derive_from"]) < 0:
            po = int(pay_off[k]) + j * C
            assert np.array_equal(to_host(r.payload[po:po + ln]), src_np[so:so + ln])
    # one flip on the wire is located in the 1 MiB-chunk layout: the master
    # (or moment) chunk that holds it, plus the derived param chunk when the
    # flipped master rounds to a different bf16 value
    sent = [k for k in range(len(t)) if int(t[k]["derive_from"]) < 0]
    starts = np.array([int(pay_off[k]) for k in sent], np.int64)
    bit = int(rng.integers(0, pb * 8))
    byte = bit // 8
    k = sent[int(np.searchsorted(starts, byte, side="right") - 1)]
    off = byte - int(pay_off[k])
    exp = {int(base[k]) + off // C}
    derived = [d for d in range(len(t)) if int(t[d]["derive_from"]) == k]
    if derived:
        d, el = derived[0], off // 4
        mo = int(t[k]["src_offset"]) + 4 * el
        m = src_np[mo:mo + 4].copy()
        m[off % 4] ^= np.uint8(1 << (bit % 8))
        po = int(t[d]["src_offset"]) + 2 * el
        if W._bf16_round(m.view(np.float32)).tobytes() != src_np[po:po + 2].tobytes():
            exp.add(int(base[d]) + (2 * el) // C)
    r.payload[byte] ^= 1 << (bit % 8)
    r.unpack()
    assert r.bad_set() == exp
    assert int(r.n_bad.item()) == len(exp)


def _flips_over_entries(t, k, seed):
    """k distinct random bit flips over the table-order concatenation of the
    entries' bytes: (arena byte offsets, bit numbers, entry of each, byte
    within that entry)."""
    nb = t["numel"].astype(np.int64) * np.where(t["dtype"] == W.F32, 4, 2)
    starts = np.concatenate([[0], np.cumsum(nb)])
    pos = W.flip_positions(int(starts[-1]) * 8, k, seed).astype(np.int64)
    cat = pos // 8
    e = np.searchsorted(starts, cat, side="right") - 1
    by = t["src_offset"].astype(np.int64)[e] + (cat - starts[e])
    return by, (pos % 8).astype(np.int64), e, cat - starts[e]


@pytest.mark.timeout(900)
def test_llama70b_stage0_replica_compare_and_checksum_whole_oracle(llama70b):
    """A replica of the 70B share with 4,096 distinct random bit flips: the
    replica compare's flagged set, count and both arenas' chunk sums, and
    the checksum of the flipped replica, equal the whole oracle's on the full
    31.8 GB arenas; the flagged set is also the closed form {chunk of each
    flipped byte}."""
    w, src_np = llama70b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    donor = _upload(src_np)
    by, bit, e, off = _flips_over_entries(t, 4096, 7096)
    _, base, _, _ = cpu.plan(t, C)
    expect = {int(base[x]) + int(o) // C for x, o in zip(e, off)}
    rep_np = src_np.copy()
    np.bitwise_xor.at(rep_np, by, (np.uint8(1) << bit.astype(np.uint8)).astype(np.uint8))
    replica = _upload(rep_np)
    nc = r.n_chunks
    sa, sb = r.plan.empty_sums(), r.plan.empty_sums()
    r.verify(donor, replica, sa, sb)
    r.checksum(replica)
    torch.cuda.synchronize()
    got = r.diff_set()
    log(f"GPU compare: {len(got)} chunks differ")
    bm, nd, osa, osb = cpu.verify(t, C, src_np, rep_np, with_sums=True)
    log("oracle compare done")
    assert got == set(cpu.bitmap_to_set(bm, nc)) == expect
    assert int(r.n_diff.item()) == nd == len(expect)
    assert np.array_equal(sums_host(sa, nc), osa) and np.array_equal(sums_host(sb, nc), osb)
    ocs = cpu.checksum(t, C, rep_np)
    assert np.array_equal(sums_host(r.csum, nc), ocs)
    log(f"compare sums and checksum equal the oracle's; {len(expect)} flagged of {nc}")


@pytest.mark.timeout(900)
def test_llama8b_striped_transfer_properties(llama8b):
    """The 8B share sent as 7 stripes (one per donor over the seven xGMI
    links of a node), each packed on its own: every stripe is the slice of
    the whole pack's payload at its first chunk's offset with the whole
    pack's sums, and the assembled buffer restores the state exactly."""
    from tests.gpu_util import striped_payload, stripe_ranges

    w, src_np = llama8b
    t, C = w.table, w.chunk_bytes
    r = Restore(t, C, w.src_arena_bytes, w.dst_arena_bytes, canary=0xA5)
    src = _upload(src_np)
    r.pack(src)
    recv, sums, parts = striped_payload(r.plan, t, src, stripe_ranges(r.n_chunks, 7))
    torch.cuda.synchronize()
    log("stripes packed")
    for (a, b), off, sp, ss in parts:
        assert torch.equal(ss, r.sums[a:b]), (a, b)
        assert off is not None and torch.equal(sp, r.payload[off:off + sp.numel()]), (a, b)
    r.unpack(payload=recv, sums=sums)
    torch.cuda.synchronize()
    assert int(r.n_bad.item()) == 0 and torch.equal(r.dst, src)


@pytest.mark.timeout(900)
def test_llama8b_delta_repair(llama8b):
    """A replica of the 8B share with 4,096 random bit flips is repaired by
    re-sending only the chunks the compare flags: the delta payload and sums
    equal the oracle's for that list, nothing is flagged on arrival, and the
    replica equals the donor byte for byte."""
    import paper_2509_03047_amd.flashrestore as F

    w, src_np = llama8b
    t, C = w.table, w.chunk_bytes
    plan = F.Plan(t, C, w.src_arena_bytes, w.dst_arena_bytes)
    donor = _upload(src_np)
    replica = donor.clone()
    pos = W.flip_positions(src_np.size * 8, 4096, 4000 + 4096)
    _flip_on_device(replica, pos)
    diff, nd = plan.empty_bitmap(), plan.empty_counter()
    ids = plan.verify_replicas(donor, replica, diff, nd, sync=True).astype(np.uint32)
    _, base, _, _ = cpu.plan(t, C)
    assert set(int(x) for x in ids) == _expected_chunks(w, base, pos)
    pb = plan.delta_layout(ids)
    payload = torch.full((pb,), 0xEE, dtype=torch.uint8, device="cuda")
    sums = torch.empty(ids.size, 2, dtype=torch.int64, device="cuda")
    plan.pack_chunks(donor, ids, payload, sums)
    bad, nbad = torch.empty((ids.size + 31) // 32, dtype=torch.int32, device="cuda"), plan.empty_counter()
    flagged = plan.unpack_chunks(payload, sums, ids, replica, bad, nbad, sync=True)
    opay, osums = cpu.pack_chunks(t, C, src_np, ids)
    assert np.array_equal(to_host(payload), opay) and np.array_equal(sums_host(sums, ids.size), osums)
    assert len(flagged) == 0 and int(nbad.item()) == 0
    assert torch.equal(replica, donor)
    log(f"delta repair: {ids.size} chunks, {pb} payload bytes")
