"""The replica compare that allocates nothing (fr_verify_replicas_noalloc),
through the C ABI: on calls in a row, each smaller than the one before, its
flagged set, count and both arenas' chunk sums equal those of
fr_verify_replicas on the same inputs (bit for bit), and the flagged set is
the oracle's; a plan whose need exceeds the static scratch is refused with
nothing written."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests.gpu_util import log, to_dev  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _case(t, C, a_np, dst_bytes, n_flips, rng, with_sums, tag):
    plan = F.Plan(t, C, max(a_np.size, 16), max(dst_bytes, 16))
    b_np = a_np.copy()
    for p in rng.choice(a_np.size * 8, size=min(n_flips, a_np.size * 8), replace=False):
        b_np[p // 8] ^= np.uint8(1 << (p % 8))
    a, b = to_dev(a_np), to_dev(b_np)
    out = {}
    for name, fn in (("alloc", plan.verify_replicas), ("noalloc", plan.verify_replicas_noalloc)):
        diff = plan.empty_bitmap().fill_(0x3C3C3C3C)
        nd = plan.empty_counter().fill_(-1)
        sa = plan.empty_sums().fill_(7) if with_sums else None
        sbs = plan.empty_sums().fill_(9) if with_sums else None
        fn(a, b, diff, nd, sa, sbs)
        torch.cuda.synchronize()
        out[name] = (diff.cpu(), int(nd.item()), None if sa is None else sa.cpu(), None if sbs is None else sbs.cpu())
    x, y = out["alloc"], out["noalloc"]
    n = plan.n_chunks
    assert torch.equal(x[0], y[0]) and x[1] == y[1], tag
    if with_sums:
        assert torch.equal(x[2][:n], y[2][:n]) and torch.equal(x[3][:n], y[3][:n]), tag
    bm, nd = cpu.verify(t, C, a_np, b_np)
    assert set(F.bitmap_indices(y[0], n).tolist()) == set(cpu.bitmap_to_set(bm, n)) and y[1] == nd, tag
    log(f"{tag}: {n} chunks, {y[1]} differ")
    return n


def test_noalloc_compare_equals_the_allocating_one_on_calls_in_a_row():
    rng = np.random.default_rng(5150)
    w = W.make_workload(0)  # toy decoder: 804 chunks of 64 KiB
    big = _case(w.table, w.chunk_bytes, W.fill_state(w), w.dst_arena_bytes, 40, rng, True, "call 1, toy decoder, sums")
    for _ in range(1000):  # a scattered table of 50-799 chunks
        t, sb, db = W.random_tiny_table(rng, max_entries=6, max_numel=3000)
        if 50 <= cpu.n_chunks(t, 256) < 800:
            break
    small = _case(t, 256, W.random_tiny_state(t, sb, rng), db, 5, rng, True, "call 2, small table, sums")
    assert 0 < small < big
    # 1 MiB chunks: 16 accumulators per chunk at the compare's 4 KiB slices
    t, nb = W.state_table([("w", 300_000), ("n", 1000)])
    smaller = _case(t, 1 << 20, W.random_tiny_state(t, nb, rng), nb, 3, rng, True, "call 3, 1 MiB chunks, sums")
    assert smaller < small
    _case(t, 1 << 20, W.random_tiny_state(t, nb, rng), nb, 2, rng, False, "call 4, no sums")


def test_noalloc_refuses_a_plan_beyond_the_static_scratch():
    # one 16 MiB tensor in 16-byte chunks: 1,048,576 chunks; the flags (4 MiB)
    # fit in the 32 MiB array, the flags plus two accumulator sets (36 MiB) do not
    t = np.zeros(1, W.TABLE_DTYPE)
    t[0] = (0, 0, 4 << 20, W.F32, -1)
    plan = F.Plan(t, 16, 16 << 20, 16 << 20)
    a = torch.zeros(16 << 20, dtype=torch.uint8, device="cuda")
    b = a.clone()
    b[12345] = 1
    diff = plan.empty_bitmap().fill_(0x3C3C3C3C)
    nd = plan.empty_counter().fill_(-1)
    sa, sbs = plan.empty_sums().fill_(7), plan.empty_sums().fill_(9)
    with pytest.raises(F.FlashRestoreError) as ei:
        plan.verify_replicas_noalloc(a, b, diff, nd, sa, sbs)
    assert ei.value.status == -3
    torch.cuda.synchronize()
    assert int(nd.item()) == -1 and bool((diff == 0x3C3C3C3C).all()) and bool((sa == 7).all())
    got = plan.verify_replicas_noalloc(a, b, diff, nd, sync=True)  # without sums it fits
    assert list(got) == [12345 // 16] and int(nd.item()) == 1
