"""The chunk-size extremes the ABI allows.  C = 2^30: a chunk spans 2^18
slices and 2^14 sub-chunk accumulators, and a derived group spans two 1 GiB
master chunks (whole-oracle parity on a 1.8 GB state with ragged tails).
C = 16: 20 million chunks and slots, so the plan's slot expansion, the
finalize kernel and the 256- and 128-thread launches all loop over more
work than one grid covers."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import flashrestore as F  # noqa: E402
from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests.gpu_util import log, sums_host, to_host  # noqa: E402


@pytest.mark.timeout(600)
def test_one_gib_chunks():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    C = 1 << 30
    n = 300_000_003  # ragged: neither array is a whole number of chunks or vectors
    mb = 4 * n
    pb = 2 * n
    m_off = 0
    p_off = (mb + 15) & ~15
    x_off = p_off + ((pb + 15) & ~15)
    arena = x_off + ((4 * 1001 + 15) & ~15)
    t = F.as_table([(p_off, p_off, n, F.FR_BF16, 1), (m_off, m_off, n, F.FR_F32, -1),
                    (x_off, x_off, 1001, F.FR_F32, -1)])
    rng = np.random.default_rng(5)
    src_np = np.zeros(arena, np.uint8)
    master = src_np[m_off:m_off + mb].view(np.float32)
    rng.standard_normal(out=master, dtype=np.float32)
    src_np[p_off:p_off + pb].view(np.uint16)[:] = W._bf16_round(master)
    src_np[x_off:x_off + 4004] = rng.integers(0, 256, 4004, dtype=np.uint8)
    log("state built")
    plan = F.Plan(t, C, arena, arena)
    assert plan.n_chunks == 2 + 1 + 1
    src = torch.from_numpy(src_np).to("cuda")
    payload, sums = plan.empty_payload().fill_(0xEE), plan.empty_sums()
    dst = torch.full((arena,), 0x3C, dtype=torch.uint8, device="cuda")
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    plan.pack(src, payload, sums)
    plan.unpack(payload, sums, dst, bad, nbad)
    torch.cuda.synchronize()
    opay, osums = cpu.pack(t, C, src_np)
    log("oracle pack done")
    assert np.array_equal(sums_host(sums, plan.n_chunks), osums)
    assert np.array_equal(to_host(payload)[: opay.size], opay)
    odst = np.full(arena, 0x3C, np.uint8)
    obm, onbad = cpu.unpack(t, C, opay, osums, odst)
    assert onbad == 0 and int(nbad.item()) == 0
    assert np.array_equal(to_host(dst), odst)
    # a wire flip inside the second master chunk is located there (and in the
    # parameter chunk when the rounding changes)
    b = (C + 12345) * 8 + 3
    payload[b // 8] ^= 1 << (b % 8)
    opay[b // 8] ^= np.uint8(1 << (b % 8))
    plan.unpack(payload, sums, dst, bad, nbad)
    odst = np.full(arena, 0x3C, np.uint8)
    obm, onbad = cpu.unpack(t, C, opay, osums, odst)
    torch.cuda.synchronize()
    got = set(F.bitmap_indices(bad, plan.n_chunks).tolist())
    assert got == set(cpu.bitmap_to_set(obm, plan.n_chunks)) and 2 in got


@pytest.mark.timeout(600)
def test_twenty_million_sixteen_byte_chunks():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests.test_gpu_parity_small import _check_against_oracle

    n = 40_000_000
    # a bf16 parameter and its master, and an fp32 array with a ragged tail
    t = np.array([(0, 0, n, W.BF16, 1), (2 * n, 2 * n, n, W.F32, -1),
                  (6 * n, 6 * n, n // 2 + 3, W.F32, -1)], dtype=W.TABLE_DTYPE)
    arena = (6 * n + 4 * (n // 2 + 3) + 15) // 16 * 16
    C = 16
    assert cpu.n_chunks(t, C) == 20_000_001  # slots of the pack walk: past 65,536 x 256
    src = W.random_tiny_state(t, arena, np.random.default_rng(17))
    log("state built")
    _check_against_oracle(t, C, src, arena, arena, corrupt_rng=np.random.default_rng(18),
                          tag="C=16, 20M chunks")
    log("20M chunks: parity")
