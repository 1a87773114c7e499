"""Restore planner for DP x TP x PP layouts with ZeRO sharding (CPU only).

Checked against the plain rules in ``oracle/planner.py`` and against
properties of the layouts: every failed rank with a live replica gets a live
donor holding identical state (same tensor, pipeline and shard position),
load is spread evenly, replicas have identical tables, the shards of a slice
tile its flattened tensors exactly, each table is accepted by the plan
validator, and derived parameter ranges are exactly the master shard."""
import itertools

import numpy as np
import pytest

from oracle import cpu, planner
from paper_2509_03047_amd import flashrestore as F

LAYOUTS = [
    (1, 1, 4, 1, 0), (2, 1, 4, 1, 0), (2, 2, 4, 2, 1), (1, 2, 8, 4, 2), (2, 2, 4, 4, 3),
    (4, 1, 2, 2, 1), (1, 1, 6, 3, 3), (2, 3, 6, 2, 2), (8, 1, 1, 1, 0),
]


@pytest.mark.parametrize("tp,pp,dp,shard,stage", LAYOUTS)
def test_coords_and_donors_match_the_rules(tp, pp, dp, shard, stage):
    L = F.Layout3D(tp, pp, dp, shard, stage)
    world = tp * pp * dp
    for r in range(world):
        assert L.coords(r) == planner.coords(tp, pp, dp, shard, r)
    rng = np.random.default_rng(world * 7 + stage)
    for _ in range(40):
        failed = set(int(x) for x in rng.choice(world, size=int(rng.integers(0, world + 1)), replace=False))
        d = L.donors(failed)
        assert d == planner.donors(tp, pp, dp, shard, failed)
        for r in range(world):
            reps = planner.replicas(tp, pp, dp, shard, r)
            if r not in failed:
                assert d[r] == -1
            elif any(x not in failed for x in reps):
                assert d[r] in reps and d[r] not in failed
                c_r, c_d = L.coords(r), L.coords(d[r])
                assert (c_r[0], c_r[1], c_r[3]) == (c_d[0], c_d[1], c_d[3])
            else:
                assert d[r] == -1
        # spread: within a replica class, donor loads differ by at most one
        loads = {}
        for r in range(world):
            if d[r] >= 0:
                loads.setdefault(tuple(sorted(planner.replicas(tp, pp, dp, shard, r))), []).append(d[r])
        for cls, used in loads.items():
            live = [x for x in cls if x not in failed]
            counts = [used.count(x) for x in live]
            assert max(counts) - min(counts) <= 1


@pytest.mark.parametrize("tp,pp,dp,shard,stage", LAYOUTS)
def test_state_tables(tp, pp, dp, shard, stage):
    L = F.Layout3D(tp, pp, dp, shard, stage)
    numel = [4096, 37, 100, 65536, 3]
    world = tp * pp * dp
    tables = {}
    for r in range(world):
        t, ab = L.state_table(r, numel)
        tables[r] = (t, ab)
        info, _, _ = F.fr_layout_query(t, 256, ab, ab)  # a valid plan table
        _, _, _, s, _ = L.coords(r)
        if stage == 0:
            assert len(t) == 4 * len(numel)
            assert info["state_bytes"] == 14 * sum(numel)
            # master, m and v of every tensor are sent, each segment at a
            # 16-byte boundary (4 KiB with 4 KiB segments), the payload
            # ending 16-aligned
            for seg in (16, 4096):
                end = 0
                for n in numel:
                    for _ in range(3):
                        end = -(-end // seg) * seg + 4 * n
                got = F.fr_layout_query(t, 256, ab, ab, seg)[0]["payload_bytes"]
                assert got == -(-end // 16) * 16
        else:
            lo, hi, npad = planner.shard_range(numel, shard, s)
            e = hi - lo
            der = [k for k in range(len(t)) if t[k]["derive_from"] >= 0]
            assert len(der) == 1
            m = int(t[der[0]]["derive_from"])
            assert int(t[der[0]]["numel"]) == int(t[m]["numel"]) == e
            if stage == 3:
                assert [int(x) for x in t["numel"]] == [e, e, e, e]
            else:
                assert [int(x) for x in t["numel"]] == [lo, e, npad - hi, e, e, e]
                assert int(t[0]["numel"]) + int(t[1]["numel"]) + int(t[2]["numel"]) == npad
    # replicas hold identical tables
    for r in range(world):
        for x in planner.replicas(tp, pp, dp, shard, r):
            assert np.array_equal(tables[r][0], tables[x][0]) and tables[r][1] == tables[x][1]
    # the shards of a slice tile the padded flat range
    if stage:
        for s0 in range(shard):
            lo, hi, npad = planner.shard_range(numel, shard, s0)
            assert lo == s0 * (npad // shard) and hi - lo == npad // shard
        assert planner.shard_range(numel, shard, shard - 1)[1] == planner.shard_range(numel, shard, 0)[2]


def test_layout_errors():
    with pytest.raises(F.FlashRestoreError):
        F.Layout3D(2, 1, 4, 3, 1).coords(0)   # shard does not divide dp
    with pytest.raises(F.FlashRestoreError):
        F.Layout3D(1, 1, 4, 2, 0).coords(0)   # vanilla DP with a shard group
    with pytest.raises(F.FlashRestoreError):
        F.Layout3D(1, 1, 4, 1, 4).coords(0)   # no ZeRO stage 4
    with pytest.raises(F.FlashRestoreError):
        F.Layout3D(2, 2, 2, 1, 0).coords(8)   # rank past the world


def test_donors_into_equals_donors():
    L = F.Layout3D(2, 2, 4, 2, 1)
    failed = [0, 5, 9]
    mask = np.zeros(L.world, np.uint8)
    mask[failed] = 1
    out = np.full(L.world, 99, np.int32)
    assert L.donors_into(mask, out).tolist() == L.donors(failed)
