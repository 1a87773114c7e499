"""Randomised GPU parity campaign: random tables (1-200 entries, scattered
layouts, derived parameters), a random tile per plan, chunks of 16 B to
1 MiB, random wire corruption; whole restore, replica compare, checksum and
a delta repair of random chunks, every output against the oracle bit for
bit.  FLASHRESTORE_CAMPAIGN="tiny,mid" sets the table counts (default
2000,60; a long run: 50000,1500)."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from paper_2509_03047_amd import workloads as W  # noqa: E402

from tests import test_gpu_parity_small as T  # noqa: E402
from tests.gpu_util import log  # noqa: E402


@pytest.mark.timeout(1200)
def test_random_campaign():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    n_tiny, n_mid = (int(x) for x in os.environ.get("FLASHRESTORE_CAMPAIGN", "2000,60").split(","))
    old = os.environ.get("FLASHRESTORE_TILE")
    rng = np.random.default_rng(2509)
    try:
        for it in range(n_tiny):
            os.environ["FLASHRESTORE_TILE"] = str(int(rng.integers(0, 11)))
            t, sb, db = W.random_tiny_table(rng, max_entries=int(rng.integers(1, 12)),
                                            max_numel=int(rng.choice([50, 300, 3000])))
            C = int(rng.choice([16, 32, 64, 128, 256, 512, 1024, 4096]))
            src = W.random_tiny_state(t, sb, rng)
            tag = f"tiny {it} tile {os.environ['FLASHRESTORE_TILE']} C={C}"
            T._check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=tag)
            if it % 4 == 0:
                T._delta_against_oracle(t, C, src, sb, db, rng, tag)
            if it % 1000 == 0:
                log(f"tiny {it}/{n_tiny}")
        for it in range(n_mid):
            os.environ["FLASHRESTORE_TILE"] = str(int(rng.integers(0, 11)))
            t, sb, db = W.random_tiny_table(rng, max_entries=int(rng.integers(1, 200)),
                                            max_numel=int(rng.choice([20_000, 100_000, 400_000])))
            C = int(rng.choice([1024, 4096, 16384, 65536, 1 << 18, 1 << 20]))
            src = W.random_tiny_state(t, sb, rng)
            tag = f"mid {it} tile {os.environ['FLASHRESTORE_TILE']} C={C} entries {len(t)}"
            T._check_against_oracle(t, C, src, sb, db, corrupt_rng=rng, tag=tag)
            T._delta_against_oracle(t, C, src, sb, db, rng, tag)
            if it % 20 == 0:
                log(f"mid {it}/{n_mid}")
    finally:
        if old is None:
            os.environ.pop("FLASHRESTORE_TILE", None)
        else:
            os.environ["FLASHRESTORE_TILE"] = old
