"""Exhaustive check of the GPU's bf16 re-derivation: every one of the 2^32
fp32 bit patterns is sent as a master value, unpack rounds it on the GPU,
and the result equals the CPU oracle's rounding bit for bit (NaN reading
included)."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from oracle import cpu  # noqa: E402
from paper_2509_03047_amd import flashrestore as F  # noqa: E402

from tests.gpu_util import log, to_host  # noqa: E402


@pytest.mark.timeout(600)
def test_rne_exhaustive_2pow32():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    n = 1 << 28  # elements per block; 16 blocks cover all 2^32 patterns
    # entry 0: bf16 param derived from entry 1 (fp32 master); src == dst layout
    t = F.as_table([(0, 0, n, F.FR_BF16, 1), (2 * n, 2 * n, n, F.FR_F32, -1)])
    arena = 6 * n
    plan = F.Plan(t, 1 << 16, arena, arena)
    src = torch.zeros(arena, dtype=torch.uint8, device="cuda")
    payload = plan.empty_payload()
    sums = plan.empty_sums()
    dst = torch.empty(arena, dtype=torch.uint8, device="cuda")
    bad, nbad = plan.empty_bitmap(), plan.empty_counter()
    for blk in range(16):
        u = np.arange(blk * n, (blk + 1) * n, dtype=np.uint64).astype(np.uint32)
        src[2 * n:].copy_(torch.from_numpy(u.view(np.uint8)))
        plan.pack(src, payload, sums)
        plan.unpack(payload, sums, dst, bad, nbad)
        exp = cpu.rne_bf16_array(u)
        got = to_host(dst[: 2 * n]).view(np.uint16)
        ok = got == exp
        assert ok.all(), f"first mismatch at {hex(int(u[np.argmin(ok)]))}: gpu {hex(int(got[np.argmin(ok)]))} oracle {hex(int(exp[np.argmin(ok)]))}"
        assert np.array_equal(to_host(dst[2 * n:]), u.view(np.uint8))
        log(f"rne block {blk + 1}/16 ok")
