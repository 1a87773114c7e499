"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host logic (validation, chunk map, payload layout) matches the oracle's
plan and the documented error codes.  No compute call needs a GPU here."""
import os
import re
import subprocess

import numpy as np
import pytest
import torch

from oracle import cpu, mini
from paper_2509_03047_amd import flashrestore as F
from paper_2509_03047_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashrestore.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(fr_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_operations():
    names = declared_functions()
    for n in ("fr_plan_create", "fr_pack_state", "fr_unpack_state", "fr_verify_replicas",
              "fr_checksum_state", "fr_layout_query", "fr_strerror", "fr_abi_version"):
        assert n in names
    assert set(names) == set(F.EXPORTED)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", F.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\sT\s+(fr_\w+)$", out, flags=re.M))
    missing = set(declared_functions()) - exported
    assert not missing, missing
    # and nothing else: the host internals are hidden
    functions = set(re.findall(r"\sT\s+(\S+)$", out, flags=re.M))
    assert functions == set(declared_functions()), functions - set(declared_functions())
    for n in declared_functions():
        assert getattr(F._lib, n) is not None


def test_library_is_gfx950_only():
    """The embedded device code targets gfx950 and nothing else."""
    blob = open(F.LIB_PATH, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa--(gfx[0-9a-z]+)", blob))
    assert targets == {b"gfx950"}, targets


def test_version_and_strerror():
    assert F.fr_abi_version() == 6
    msgs = {c: F.fr_strerror(c) for c in range(-7, 1)}
    assert msgs[0] == "ok" and len(set(msgs.values())) == 8
    assert F.fr_strerror(-99) == "unknown status"


def _check_layout(t, C, sb, db, seg=16):
    info, pay, base = F.fr_layout_query(t, C, sb, db, seg)
    nch, obase, opay, opb = cpu.plan(t, C, seg)
    assert info["segment_align"] == seg
    assert info["payload_bytes"] == opb
    assert info["n_chunks"] == int(obase[-1])
    assert info["bitmap_words"] == (int(obase[-1]) + 31) // 32
    assert info["device"] == -1 and info["pack_walk"] == info["unpack_walk"] == 0  # no plan
    assert np.array_equal(base, obase)
    for k in range(len(t)):
        if int(t[k]["derive_from"]) >= 0:
            assert int(pay[k]) == F.NO_PAYLOAD
        else:
            assert int(pay[k]) == int(opay[k])
    return info


@pytest.mark.parametrize("config", [0, 1, 2, 3])
def test_layout_matches_oracle_on_workloads(config):
    w = W.make_workload(config)
    info = _check_layout(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
    # 12 payload bytes per param, segments back to back
    exp = {0: (804, 44_055_552), 1: (214_684, 12_048_187_392), 3: (30_474, 27_249_082_368)}
    if config in exp:
        assert (info["n_chunks"], info["payload_bytes"]) == exp[config]
        assert info["payload_bytes"] == 12 * w.n_params
        assert info["state_bytes"] == 14 * w.n_params
    # 4 KiB segments: the toy gains 14 gaps of 3 KiB after its 1 KiB norm
    # arrays; the 8B and 70B shares, whose tensors are whole multiples of
    # 4 KiB, keep the same payload
    info4 = _check_layout(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes, 4096)
    exp4 = {0: 44_098_560, 1: 12_048_187_392, 3: 27_249_082_368}
    if config in exp4:
        assert info4["payload_bytes"] == exp4[config]


def test_layout_matches_both_oracles_on_random_tables():
    rng = np.random.default_rng(41)
    for _ in range(300):
        t, sb, db = W.random_tiny_table(rng)
        C = int(rng.choice([16, 32, 64, 256, 4096]))
        seg = int(rng.choice([16, 32, 256, 4096, 1 << 20]))
        _check_layout(t, C, sb, db, seg)
        _, mbase, mpay, mpb = mini.plan(t, C, seg)
        info, pay, base = F.fr_layout_query(t, C, sb, db, seg)
        assert list(base) == mbase and info["payload_bytes"] == mpb


def _rows():
    # two bf16/fp32 pairs, properly derived, 16-aligned, inside 4 KiB arenas
    return [
        [0, 0, 10, 2, 1],
        [32, 32, 10, 1, -1],
        [80, 80, 7, 1, -1],
    ]


def _q(rows, C=64, sb=4096, db=4096):
    try:
        F.fr_layout_query(rows, C, sb, db)
        return 0
    except F.FlashRestoreError as e:
        return e.status


def test_valid_baseline_table():
    assert _q(_rows()) == 0


@pytest.mark.parametrize(
    "mutate, code",
    [
        (lambda r: r[0].__setitem__(3, 3), -1),                 # bad dtype
        (lambda r: r[0].__setitem__(4, 5), -1),                 # derive_from out of range
        (lambda r: r[0].__setitem__(4, 0), -1),                 # derives from itself
        (lambda r: r[0].__setitem__(3, 1), -1),                 # derived entry not bf16
        (lambda r: r[1].__setitem__(2, 11), -1),                # numel mismatch with master
        (lambda r: r[1].__setitem__(3, 2), -1),                 # master not fp32
        (lambda r: r.append([200, 200, 10, 2, 1]), -1),        # second derivation of one master
        (lambda r: r[2].__setitem__(4, 0), -1),                 # derives from a derived entry
        (lambda r: r[1].__setitem__(0, 40), -2),                # src offset % 16
        (lambda r: r[1].__setitem__(1, 8), -2),                 # dst offset % 16
        (lambda r: r[2].__setitem__(0, 4080), -3),              # past the sender arena
        (lambda r: r[2].__setitem__(1, 4080), -3),              # past the receiver arena
        (lambda r: r[2].__setitem__(2, 1 << 62), -3),           # absurd numel
        (lambda r: r[2].__setitem__(1, 32), -4),                # receiver ranges overlap
    ],
)
def test_table_errors(mutate, code):
    rows = _rows()
    mutate(rows)
    assert _q(rows) == code


def test_sender_ranges_may_overlap_and_empty_entries_are_fine():
    rows = _rows()
    rows[2][0] = 32  # reads the same bytes as entry 1
    assert _q(rows) == 0
    rows.append([4096, 4096, 0, 1, -1])  # empty entry exactly at the arena end
    assert _q(rows) == 0
    assert _q([]) == 0


@pytest.mark.parametrize("C, code", [(0, -1), (8, -1), (48, -1), (1 << 31, -1), (16, 0), (1 << 30, 0)])
def test_chunk_size_rule(C, code):
    assert _q(_rows(), C=C) == code


@pytest.mark.parametrize("seg, code", [(0, -1), (8, -1), (48, -1), (1 << 21, -1), (16, 0), (4096, 0),
                                       (1 << 20, 0)])
def test_segment_alignment_rule(seg, code):
    try:
        F.fr_layout_query(_rows(), 64, 4096, 4096, seg)
        rc = 0
    except F.FlashRestoreError as e:
        rc = e.status
    assert rc == code


TILE_KEYS = ("tile_pack", "tile_unpack", "tile_verify", "tile_checksum")


def _tiles(C):
    info, _, _ = F.fr_layout_query(_rows(), C, 1 << 20, 1 << 20)
    return tuple(info[k] for k in TILE_KEYS)


def _clear_tile_env(monkeypatch):
    for k in list(os.environ):
        if k.startswith("FLASHRESTORE_TILE"):
            monkeypatch.delenv(k)


@pytest.mark.parametrize("C, want", [(16, (4, 7, 7, 4)), (1024, (4, 7, 7, 4)), (2048, (4, 6, 7, 4)),
                                     (4096, (4, 5, 5, 4)), (8192, (4, 5, 5, 9)), (16384, (4, 5, 5, 3)),
                                     (1 << 30, (4, 5, 5, 3))])
def test_tiles_follow_the_chunk_size(C, want, monkeypatch):
    """Unset, each operation's tile follows the chunk size (pack 64x4 = 4;
    unpack 64x1 = 7 up to 1 KiB, 64x2 = 6 at 2 KiB, else 128x2 = 5; compare
    64x1 up to 2 KiB, else 128x2; checksum 64x4 up to 4 KiB, 128x4 = 9 at
    8 KiB, else 256x4 = 3)."""
    _clear_tile_env(monkeypatch)
    assert _tiles(C) == want


def test_tile_variables_override_the_chunk_size_rule(monkeypatch):
    _clear_tile_env(monkeypatch)
    monkeypatch.setenv("FLASHRESTORE_TILE", "9")
    assert _tiles(1024) == (9, 9, 9, 9)
    monkeypatch.setenv("FLASHRESTORE_TILE_CHECKSUM", "2")
    assert _tiles(1024) == (9, 9, 9, 2)
    monkeypatch.delenv("FLASHRESTORE_TILE")
    monkeypatch.setenv("FLASHRESTORE_TILE_UNPACK", "0")
    assert _tiles(1024) == (4, 0, 7, 2)
    assert _tiles(1 << 20) == (4, 0, 5, 2)


def test_chunk_id_limit():
    # 2^32 chunks of 16 bytes would overflow 32-bit chunk ids
    rows = [[0, 0, 1 << 34, 1, -1]]
    assert _q(rows, C=16, sb=1 << 37, db=1 << 37) == -3
    assert _q(rows, C=1 << 20, sb=1 << 37, db=1 << 37) == 0


def test_plan_create_without_a_gpu_reports_a_device_error():
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(F.FlashRestoreError) as ei:
        F.Plan(_rows(), 64, 4096, 4096)
    assert ei.value.status == -6


def test_binding_refuses_to_run_without_the_library(tmp_path, monkeypatch):
    """The product path has no fallback: a missing library is an import error."""
    import importlib.util

    spec = importlib.util.spec_from_file_location("fr_copy", F.__file__)
    mod = importlib.util.module_from_spec(spec)
    monkeypatch.setattr(os.path, "exists", lambda p: False if p.endswith("libflashrestore.so") else True)
    with pytest.raises(ImportError):
        spec.loader.exec_module(mod)


def test_bench_refuses_more_than_one_gpu():
    """One GPU only: bench.py with --gpus above 1 exits with a message before
    touching any device."""
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    p = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr and p.stdout == ""
