"""End-to-end restore of failed ranks in a DP x TP x PP layout with ZeRO
sharding, on one GPU: every rank's state arena is built from one consistent
global state, failed ranks are restored by packing their donor's arena and
unpacking into a fresh one, and each restored arena equals the failed rank's
own bit for bit with no chunk flagged."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

NUMEL = [65536, 4096, 1000, 30000, 7]


def _slice_state(rng, n):
    master = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    return master, m, v


def _arena(L, rank, stage, states):
    """The rank's arena built from its slice's global state and its table."""
    t, ab = L.state_table(rank, NUMEL)
    tp_i, pp_i, _, s, _ = L.coords(rank)
    master, m, v = states[(tp_i, pp_i)]
    a = np.zeros(ab, np.uint8)

    def put(k, arr):
        o = int(t[k]["src_offset"])
        b = np.ascontiguousarray(arr).view(np.uint8)
        a[o:o + b.size] = b

    if stage == 0:
        off = 0
        for k, n in enumerate(NUMEL):
            mk = master[off:off + n]
            put(4 * k, W._bf16_round(mk))
            put(4 * k + 1, mk)
            put(4 * k + 2, m[off:off + n])
            put(4 * k + 3, v[off:off + n])
            off += n
    else:
        e = int(t[-1]["numel"])
        lo, hi = s * e, (s + 1) * e
        params = W._bf16_round(master)
        if stage == 3:
            put(0, params[lo:hi])
            put(1, master[lo:hi])
            put(2, m[lo:hi])
            put(3, v[lo:hi])
        else:
            put(0, params[:lo])
            put(1, params[lo:hi])
            put(2, params[hi:])
            put(3, master[lo:hi])
            put(4, m[lo:hi])
            put(5, v[lo:hi])
    return t, a


@pytest.mark.parametrize("tp,pp,dp,shard,stage", [(2, 2, 4, 1, 0), (2, 2, 4, 2, 1), (1, 2, 8, 4, 2), (2, 1, 6, 3, 3)])
def test_restore_failed_ranks_from_their_donors(tp, pp, dp, shard, stage):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L = F.Layout3D(tp, pp, dp, shard, stage)
    world = tp * pp * dp
    rng = np.random.default_rng(world + 31 * stage)
    n = sum(NUMEL)
    npad = -(-n // (8 * shard)) * (8 * shard) if stage else n
    states = {}
    for tp_i in range(tp):
        for pp_i in range(pp):
            master, m, v = _slice_state(rng, npad)
            if stage:  # padding elements hold zeros in every array
                master[n:] = 0
                m[n:] = 0
                v[n:] = 0
            states[(tp_i, pp_i)] = (master, m, v)
    failed = set(int(x) for x in rng.choice(world, size=max(1, world // 4), replace=False))
    donors = L.donors(failed)
    restored = 0
    for r in sorted(failed):
        if donors[r] < 0:
            continue
        t, expect = _arena(L, r, stage, states)
        t_d, donor_np = _arena(L, donors[r], stage, states)
        assert np.array_equal(t, t_d) and np.array_equal(expect, donor_np)  # replicas agree
        plan = F.Plan(t, 4096, expect.size, expect.size)
        src = torch.from_numpy(donor_np).to("cuda")
        dst = torch.full((expect.size,), 0xEE, dtype=torch.uint8, device="cuda")
        payload, sums = plan.empty_payload(), plan.empty_sums()
        bad, nbad = plan.empty_bitmap(), plan.empty_counter()
        plan.pack(src, payload, sums)
        plan.unpack(payload, sums, dst, bad, nbad)
        torch.cuda.synchronize()
        assert int(nbad.item()) == 0
        got = dst.cpu().numpy()
        inside = np.zeros(expect.size, bool)
        for e in t:
            o, nb = int(e["dst_offset"]), int(e["numel"]) * (4 if int(e["dtype"]) == 1 else 2)
            inside[o:o + nb] = True
        assert np.array_equal(got[inside], expect[inside]), f"rank {r} from {donors[r]}"
        assert (got[~inside] == 0xEE).all()  # alignment gaps are never written
        restored += 1
    assert restored >= 1
