"""Randomised GPU parity campaign: random tables (1-200 entries, scattered
layouts, derived parameters), each under a random launch configuration
(one tile for all, or tiles chosen by chunk size, sometimes one operation
with its own, the pack / unpack / compare / checksum walks, absorbing last slices,
buffer loads, walk orders, grid and delta grid caps) and a random payload
segment alignment, chunks of 16 B to 1 MiB, random wire corruption; whole
restore, replica compare, checksum and (at 16-byte segments) a delta repair
of random chunks, every output against the oracle bit for bit.  Results
never depend on the launch configuration; this checks that over
combinations the other tests do not enumerate.  FLASHRESTORE_CAMPAIGN=
"tiny,mid" sets the table counts (default 2000,60; a long run:
50000,1500)."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests import test_gpu_parity_small as T  # noqa: E402
from tests.gpu_util import log  # noqa: E402

KNOBS = ("FLASHRESTORE_TILE", "FLASHRESTORE_LINE_PACK", "FLASHRESTORE_LINE_UNPACK",
         "FLASHRESTORE_LINE_VERIFY", "FLASHRESTORE_LINE_CHECKSUM", "FLASHRESTORE_ABSORB_PACK",
         "FLASHRESTORE_ABSORB_UNPACK", "FLASHRESTORE_BUF_PACK", "FLASHRESTORE_BUF_UNPACK",
         "FLASHRESTORE_BUF_VERIFY", "FLASHRESTORE_BUF_CHECKSUM", "FLASHRESTORE_ORDER_VERIFY",
         "FLASHRESTORE_ORDER_CHECKSUM", "FLASHRESTORE_MAX_GRID", "FLASHRESTORE_DELTA_GRID",
         "FLASHRESTORE_LINE", "FLASHRESTORE_TILE_PACK", "FLASHRESTORE_TILE_UNPACK",
         "FLASHRESTORE_TILE_VERIFY", "FLASHRESTORE_TILE_CHECKSUM")


def _random_knobs(rng) -> str:
    for k in KNOBS:
        os.environ.pop(k, None)
    tile = int(rng.integers(-4, 11))  # negative: unset, each tile chosen by the chunk size
    if tile >= 0:
        os.environ["FLASHRESTORE_TILE"] = str(tile)
    if rng.random() < 0.25:  # one operation with a tile of its own
        os.environ[str(rng.choice(KNOBS[16:]))] = str(int(rng.integers(0, 11)))
    for k in ("FLASHRESTORE_LINE_PACK", "FLASHRESTORE_LINE_UNPACK"):
        v = int(rng.integers(-1, 5))  # -1: unset, the walk chosen by the table
        if v >= 0:
            os.environ[k] = str(v)
    for k in KNOBS[3:13]:
        if rng.random() < 0.5:
            os.environ[k] = str(int(rng.integers(0, 2)))
    os.environ["FLASHRESTORE_MAX_GRID"] = str(int(rng.choice([0, 0, 0, 1, 7, 300])))
    os.environ["FLASHRESTORE_DELTA_GRID"] = str(int(rng.choice([65536, 65536, 1, 13])))
    return " ".join(f"{k[13:]}={os.environ[k]}" for k in KNOBS if k in os.environ)


@pytest.mark.timeout(1200)
def test_random_campaign():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    n_tiny, n_mid = (int(x) for x in os.environ.get("FLASHRESTORE_CAMPAIGN", "2000,60").split(","))
    old = {k: os.environ.get(k) for k in KNOBS}
    rng = np.random.default_rng(2509)
    try:
        for it in range(n_tiny):
            desc = _random_knobs(rng)
            t, sb, db = W.random_tiny_table(rng, max_entries=int(rng.integers(1, 12)),
                                            max_numel=int(rng.choice([50, 300, 3000])))
            C = int(rng.choice([16, 32, 64, 128, 256, 512, 1024, 4096]))
            seg = int(rng.choice([16, 16, 16, 32, 64, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            tag = f"tiny {it} C={C} seg={seg} {desc}"
            T._check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=tag, seg=seg)
            if it % 4 == 0 and seg == 16:
                T._delta_against_oracle(t, C, src, sb, db, rng, tag)
            if it % 1000 == 0:
                log(f"tiny {it}/{n_tiny}")
        for it in range(n_mid):
            desc = _random_knobs(rng)
            t, sb, db = W.random_tiny_table(rng, max_entries=int(rng.integers(1, 200)),
                                            max_numel=int(rng.choice([20_000, 100_000, 400_000])))
            C = int(rng.choice([1024, 4096, 16384, 65536, 1 << 18, 1 << 20]))
            seg = int(rng.choice([16, 16, 64, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            tag = f"mid {it} C={C} seg={seg} entries {len(t)} {desc}"
            T._check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=tag, seg=seg)
            if seg == 16:
                T._delta_against_oracle(t, C, src, sb, db, rng, tag)
            if it % 20 == 0:
                log(f"mid {it}/{n_mid}")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
