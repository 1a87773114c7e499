"""Seeded synthetic workloads: descriptor tables and state bytes.

This module is the only code that the GPU path and the CPU oracle share, and
it holds none of the restore method's arithmetic: no chunking, no checksum,
no payload layout and no hand-written rounding.  It builds

* the tensor lists of the five restore workloads (a toy decoder, one rank's
  share of a Llama-3-8B-shaped state under tensor parallel 8, a 20,000-entry
  descriptor stress table, one rank's share of a Llama-3-70B-shaped state
  under TP 8 x PP 4, and a replica-compare pair of the 8B share),
* the 32-byte tensor-descriptor table that both the library and the oracle
  take as input (``TABLE_DTYPE``),
* the state bytes, drawn from seeded numpy generators, and
* seeded sets of distinct bit positions for flip injection.

The training state restored in data-parallel recovery is a rank's model
state: parameters plus optimizer state (Section II, "model state"; Section
III-E, restoration from a data-parallel replica).  Each logical tensor here
carries four arrays: a bf16 parameter, an fp32 master copy, and fp32 Adam
first and second moments.  The parameter is the master rounded to bf16 by
torch's CPU cast (round to nearest even for the finite values drawn here);
no rounding code of this project is used to make inputs.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

# Descriptor layout: 32 bytes, little endian, no padding.
#   src_offset  byte offset of the tensor in the sender (or replica) arena
#   dst_offset  byte offset of the tensor in the receiver arena
#   numel       element count (0 allowed)
#   dtype       1 = fp32, 2 = bf16
#   derive_from -1, or the index of the fp32 master this bf16 tensor is
#               rounded from
TABLE_DTYPE = np.dtype(
    [
        ("src_offset", "<u8"),
        ("dst_offset", "<u8"),
        ("numel", "<u8"),
        ("dtype", "<u4"),
        ("derive_from", "<i4"),
    ]
)
assert TABLE_DTYPE.itemsize == 32

F32 = 1
BF16 = 2
ESIZE = {F32: 4, BF16: 2}

# The four arrays of one logical tensor, in table order, with the standard
# deviation each is drawn with (v is the absolute value of its draw).
STATE_ARRAYS = ("param", "master", "m", "v")
SIGMA = {"master": 0.02, "m": 1e-3, "v": 1e-6}


@dataclass
class Workload:
    """A descriptor table plus the sizes of the arenas it addresses."""

    name: str
    table: np.ndarray  # TABLE_DTYPE
    chunk_bytes: int
    src_arena_bytes: int
    dst_arena_bytes: int
    tensors: list  # (name, numel) of the logical tensors, or None
    seed: int

    @property
    def n_params(self) -> int:
        if self.tensors is None:
            return int(self.table["numel"].sum())
        return int(sum(n for _, n in self.tensors))

    @property
    def state_bytes(self) -> int:
        """Bytes of tensor data in the table (gaps between tensors excluded)."""
        es = np.where(self.table["dtype"] == F32, 4, 2).astype(np.uint64)
        return int((self.table["numel"] * es).sum())


# ---------------------------------------------------------------- tensor lists


def toy_decoder_tensors():
    """2 layers, d=256, ffn=1024, vocab 8192, tied embedding, 2-matrix FFN."""
    d, ffn, vocab = 256, 1024, 8192
    t = [("embed", vocab * d)]
    for l in range(2):
        t += [
            (f"l{l}.attn_norm", d),
            (f"l{l}.wqkv", d * 3 * d),
            (f"l{l}.wo", d * d),
            (f"l{l}.ffn_norm", d),
            (f"l{l}.w1", d * ffn),
            (f"l{l}.w2", ffn * d),
        ]
    t.append(("final_norm", d))
    return t


def _llama_rank_share(layers, hidden, n_q, n_kv, ffn, vocab, tp, with_head):
    """One tensor-parallel rank's share of a Llama-shaped decoder.

    Column-parallel (qkv, gate+up) and row-parallel (o, down) weights are split
    by ``tp``; the vocabulary is split by ``tp``; RMSNorm weights are
    replicated.  Gate and up projections are fused into one fc1 matrix.
    """
    head = hidden // n_q
    q_loc, kv_loc = n_q * head // tp, n_kv * head // tp
    ffn_loc, vocab_loc = ffn // tp, -(-vocab // tp)
    t = [("embed", vocab_loc * hidden)]
    for l in range(layers):
        t += [
            (f"l{l}.attn_norm", hidden),
            (f"l{l}.wqkv", hidden * (q_loc + 2 * kv_loc)),
            (f"l{l}.wo", q_loc * hidden),
            (f"l{l}.ffn_norm", hidden),
            (f"l{l}.fc1", hidden * 2 * ffn_loc),
            (f"l{l}.fc2", ffn_loc * hidden),
        ]
    if with_head:
        t += [("final_norm", hidden), ("lm_head", vocab_loc * hidden)]
    return t


def llama3_8b_tp8_tensors():
    """Llama-3-8B shape, TP=8: 32 layers, hidden 4096, 32q/8kv, ffn 14336, vocab 128256."""
    return _llama_rank_share(32, 4096, 32, 8, 14336, 128256, 8, with_head=True)


def llama3_70b_tp8_pp4_stage0_tensors():
    """Llama-3-70B shape, TP=8 x PP=4, first stage: embedding + layers 0..19."""
    return _llama_rank_share(20, 8192, 64, 8, 28672, 128256, 8, with_head=False)


# ---------------------------------------------------------------- tables


def state_table(tensors):
    """Four entries per logical tensor, contiguous in table order, same layout
    on both sides.  Returns (table, arena_bytes)."""
    rows = []
    off = 0
    for _, n in tensors:
        base = len(rows)
        for kind in STATE_ARRAYS:
            dt = BF16 if kind == "param" else F32
            nbytes = n * ESIZE[dt]
            der = base + 1 if kind == "param" else -1
            rows.append((off, off, n, dt, der))
            off += -(-nbytes // 16) * 16
    table = np.array(rows, dtype=TABLE_DTYPE)
    return table, off


def make_workload(config: int) -> Workload:
    """Tables of the five restore workloads.

    0  toy decoder, 64 KiB chunks
    1  Llama-3-8B TP=8 rank share, 64 KiB chunks
    2  20,000-entry descriptor stress, 16 KiB chunks
    3  Llama-3-70B TP=8 x PP=4 first-stage share, 1 MiB chunks
    4  replica compare on the config-1 table (values: two copies + flips)
    """
    if config in (0, 1, 3, 4):
        tensors = {
            0: toy_decoder_tensors,
            1: llama3_8b_tp8_tensors,
            3: llama3_70b_tp8_pp4_stage0_tensors,
            4: llama3_8b_tp8_tensors,
        }[config]()
        table, nb = state_table(tensors)
        c = {0: 1 << 16, 1: 1 << 16, 3: 1 << 20, 4: 1 << 16}[config]
        names = {
            0: "toy-decoder-2L-d256",
            1: "llama3-8b-tp8-rank-state",
            3: "llama3-70b-tp8pp4-stage0-rank-state",
            4: "llama3-8b-tp8-replica-pair",
        }
        return Workload(names[config], table, c, nb, nb, tensors, config)
    if config == 2:
        return stress_workload(seed=2)
    raise ValueError(f"no workload {config}")


def _scatter_layout(nbytes, rng):
    """Shuffled placement with random 16-byte-multiple gaps (0..255 * 16 B)."""
    n = len(nbytes)
    order = rng.permutation(n)
    gaps = rng.integers(0, 256, size=n, dtype=np.int64) * 16
    off = np.zeros(n, dtype=np.uint64)
    pos = 0
    for i, k in enumerate(order):
        pos += int(gaps[i])
        off[k] = pos
        pos += -(-int(nbytes[k]) // 16) * 16
    return off, pos


def stress_workload(seed=2, n_entries=20000, lo=256, hi=1 << 20, chunk_bytes=1 << 14):
    """Descriptor-overhead stress: many fp32/bf16 tensors, log-uniform sizes,
    independent shuffled src and dst layouts with gaps, no derived entries."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    dts = np.where(rng.random(n_entries) < 0.5, F32, BF16).astype(np.uint32)
    u = rng.random(n_entries)
    numel = np.floor(lo * (hi / lo) ** u).astype(np.uint64)
    nbytes = numel * np.where(dts == F32, 4, 2).astype(np.uint64)
    src_off, src_bytes = _scatter_layout(nbytes, rng)
    drng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed + 1000, 0])))
    dst_off, dst_bytes = _scatter_layout(nbytes, drng)
    table = np.zeros(n_entries, dtype=TABLE_DTYPE)
    table["src_offset"] = src_off
    table["dst_offset"] = dst_off
    table["numel"] = numel
    table["dtype"] = dts
    table["derive_from"] = -1
    return Workload("descriptor-stress-20k", table, chunk_bytes, src_bytes, dst_bytes, None, seed)


# ---------------------------------------------------------------- values


def _rng(seed, *key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *key])))


def _bf16_round(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of fp32 values by torch's CPU cast (uint16 array)."""
    import torch

    x = np.ascontiguousarray(x, dtype=np.float32)
    if not x.flags.writeable:
        x = x.copy()
    t = torch.from_numpy(x).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _threads():
    return max(1, min(16, int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))))


def fill_state(w: Workload, arena: np.ndarray | None = None, threads: int | None = None) -> np.ndarray:
    """Draw the sender state bytes of ``w`` into a uint8 arena (gaps = 0).

    Every array of every logical tensor has its own generator keyed by
    (seed, tensor index, array), so the bytes do not depend on thread count.
    """
    if arena is None:
        arena = np.zeros(w.src_arena_bytes, dtype=np.uint8)
    if arena.dtype != np.uint8 or arena.size < w.src_arena_bytes:
        raise ValueError("arena must be a uint8 array of at least src_arena_bytes")
    t = w.table
    jobs = []
    if w.tensors is not None:
        for i in range(len(w.tensors)):
            jobs.append(("state", i))
    else:
        for k in range(len(t)):
            jobs.append(("generic", k))

    def run(job):
        kind, i = job
        if kind == "state":
            p, mst, m, v = (t[4 * i + j] for j in range(4))
            n = int(mst["numel"])

            def f32(e):
                o = int(e["src_offset"])
                return arena[o : o + 4 * n].view(np.float32)

            mv = f32(mst)
            _rng(w.seed, i, 1).standard_normal(out=mv, dtype=np.float32)
            mv *= np.float32(SIGMA["master"])
            po = int(p["src_offset"])
            arena[po : po + 2 * n].view(np.uint16)[:] = _bf16_round(mv)
            mm = f32(m)
            _rng(w.seed, i, 2).standard_normal(out=mm, dtype=np.float32)
            mm *= np.float32(SIGMA["m"])
            vv = f32(v)
            _rng(w.seed, i, 3).standard_normal(out=vv, dtype=np.float32)
            vv *= np.float32(SIGMA["v"])
            vv.view(np.uint32)[:] &= np.uint32(0x7FFFFFFF)
        else:
            e = t[i]
            n, o = int(e["numel"]), int(e["src_offset"])
            x = np.empty(n, dtype=np.float32)
            _rng(w.seed, i, 0).standard_normal(out=x, dtype=np.float32)
            if int(e["dtype"]) == F32:
                arena[o : o + 4 * n].view(np.float32)[:] = x
            else:
                arena[o : o + 2 * n].view(np.uint16)[:] = _bf16_round(x)
        return 0

    nt = threads or _threads()
    if nt == 1:
        for j in jobs:
            run(j)
    else:
        with ThreadPoolExecutor(nt) as ex:
            list(ex.map(run, jobs))
    return arena


def flip_positions(n_bits_total: int, k: int, seed: int) -> np.ndarray:
    """k distinct bit positions drawn uniformly from [0, n_bits_total), sorted."""
    rng = _rng(seed, 0)
    if k == 0:
        return np.zeros(0, dtype=np.uint64)
    picked = set()
    while len(picked) < k:
        need = k - len(picked)
        for p in rng.integers(0, n_bits_total, size=2 * need, dtype=np.uint64):
            picked.add(int(p))
            if len(picked) == k:
                break
    return np.array(sorted(picked), dtype=np.uint64)


def apply_flips(arena: np.ndarray, bit_positions: np.ndarray) -> None:
    """XOR the given bit positions (byte = p // 8, bit = p % 8) in place."""
    for p in bit_positions:
        p = int(p)
        arena[p >> 3] ^= np.uint8(1 << (p & 7))


def random_tiny_table(rng: np.random.Generator, max_entries=6, max_numel=300, allow_derive=True):
    """A small random descriptor table for brute-force comparisons.

    Entries get random dtypes, sizes 0..max_numel, shuffled src/dst placement
    with random 16-byte gaps; some bf16 entries derive from an fp32 master of
    equal length that no other entry derives from.
    """
    n = int(rng.integers(1, max_entries + 1))
    numel = rng.integers(0, max_numel + 1, size=n).astype(np.uint64)
    dts = np.where(rng.random(n) < 0.5, F32, BF16).astype(np.uint32)
    der = np.full(n, -1, dtype=np.int32)
    if allow_derive and n >= 2:
        used = set()
        for k in range(n):
            if rng.random() < 0.4:
                cands = [s for s in range(n) if s != k and dts[s] == F32 and der[s] == -1 and s not in used]
                if cands and k not in used:
                    s = int(rng.choice(cands))
                    dts[k] = BF16
                    numel[k] = numel[s]
                    der[k] = s
                    used.add(s)
    nbytes = numel * np.where(dts == F32, 4, 2).astype(np.uint64)
    src_off, src_bytes = _scatter_layout(nbytes, rng)
    dst_off, dst_bytes = _scatter_layout(nbytes, rng)
    table = np.zeros(n, dtype=TABLE_DTYPE)
    table["src_offset"] = src_off
    table["dst_offset"] = dst_off
    table["numel"] = numel
    table["dtype"] = dts
    table["derive_from"] = der
    return table, int(src_bytes), int(dst_bytes)


def random_tiny_state(table: np.ndarray, arena_bytes: int, rng: np.random.Generator) -> np.ndarray:
    """Random bytes for every entry; derived bf16 entries = cast of their master."""
    a = np.zeros(max(arena_bytes, 0), dtype=np.uint8)
    for k in range(len(table)):
        e = table[k]
        nb = int(e["numel"]) * ESIZE[int(e["dtype"])]
        o = int(e["src_offset"])
        if int(e["dtype"]) == F32:
            x = rng.standard_normal(int(e["numel"])).astype(np.float32)
            a[o : o + nb].view(np.float32)[:] = x
        else:
            a[o : o + nb] = rng.integers(0, 256, size=nb, dtype=np.uint8)
    for k in range(len(table)):
        e = table[k]
        s = int(e["derive_from"])
        if s >= 0:
            n = int(e["numel"])
            so, o = int(table[s]["src_offset"]), int(e["src_offset"])
            a[o : o + 2 * n].view(np.uint16)[:] = _bf16_round(a[so : so + 4 * n].view(np.float32))
    return a
