"""A whole restore step captured in a HIP graph (the operations are kernel
launches only: no memsets, no host work on the stream) and replayed several
times, with eager work and synchronisation between replays; every replay is
checked against the eager result."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402


def test_captured_restore_step_replays_correctly():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make_workload(0)
    src_np = W.fill_state(w)
    plan = F.Plan(w.table, w.chunk_bytes, w.src_arena_bytes, w.dst_arena_bytes)
    src = torch.from_numpy(src_np).to("cuda")
    payload, sums = plan.empty_payload(), plan.empty_sums()
    dst = torch.zeros(w.dst_arena_bytes, dtype=torch.uint8, device="cuda")
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    diff, ndiff = plan.empty_bitmap(), plan.empty_counter()
    csum = plan.empty_sums()

    def step():
        plan.pack(src, payload, sums)
        plan.unpack(payload, sums, dst, bad, nbad)
        plan.verify_replicas(src, dst, diff, ndiff)
        plan.checksum_state(dst, csum)

    # eager reference of the unmodified state
    step()
    torch.cuda.synchronize()
    ref = (payload.clone(), sums.clone(), dst.clone(), csum.clone())

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on the capture stream
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    rng = np.random.default_rng(3)
    for rep in range(4):
        # eager work between replays: perturb the donor, then restore it later
        flip = int(rng.integers(0, src.numel()))
        src[flip] ^= 0x10
        dst.fill_(0x77)
        nbad.fill_(99)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        # the captured step saw the perturbed donor: check against eager
        exp_payload, exp_sums = plan.empty_payload(), plan.empty_sums()
        plan.pack(src, exp_payload, exp_sums)
        torch.cuda.synchronize()
        assert torch.equal(payload, exp_payload) and torch.equal(sums, exp_sums), rep
        assert torch.equal(dst, src) and int(nbad.item()) == 0 and int(ndiff.item()) == 0
        assert torch.equal(csum, sums)
        src[flip] ^= 0x10  # undo
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(payload, ref[0]) and torch.equal(sums, ref[1])
    assert torch.equal(dst, ref[2]) and torch.equal(csum, ref[3])
