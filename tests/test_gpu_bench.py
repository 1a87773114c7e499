"""bench.py end to end on small runs: the one JSON line it prints carries the
contract's fields, and the pass, the delta repair and the control-plane
checks all report success (toy decoder; descriptor stress, whose receiver
layout differs from the sender's)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("config,extra", [(0, ["--cpu-sample-bytes", "20000000"]), (2, ["--no-cpu-baseline"])])
def test_bench_json_line(config, extra):
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--config", str(config),
                        "--steps", "2", "--warmup", "1", *extra],
                       cwd=ROOT, capture_output=True, text=True, timeout=500)
    assert p.returncode == 0, p.stderr[-3000:]
    lines = [ln for ln in p.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "ops"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["higher_is_better"] is True
    assert d["value"] > 0 and d["config"]["workload"]
    # value is the restore rate: state bytes over pack + unpack time
    restore_ms = d["ops"]["pack"]["ms"] + d["ops"]["unpack"]["ms"]
    assert abs(d["value"] - d["config"]["state_bytes"] / (restore_ms * 1e-3) / 1e9) < 0.01 * d["value"]
    assert d["step_gbs"] < d["value"]
    ce = d["ceilings"]
    assert ce["copy_gbs"] > 0 and ce["read_gbs"] > 0 and ce["write_gbs"] > 0
    for op, o in d["ops"].items():
        assert o["ceiling"] in ("copy", "read")
        assert abs(o["frac_of_ceiling"] - o["hbm_gbs"] / ce[o["ceiling"] + "_gbs"]) < 1e-3
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    # the stress table's chunks start inside lines on both sides written: tile walks
    walks = d["config"]["walks"]
    if config == 2:
        assert walks == {"pack": "tiles of the side written", "unpack": "tiles of the side written"}
        assert r["kernel"] in ("k_pack_blocks", "k_unpack_blocks", "k_verify", "k_pack")
    # 64 KiB and 16 KiB chunks keep every operation's default tile
    assert d["config"]["tiles"] == {"pack": "64x4", "unpack": "128x2", "verify": "128x2", "checksum": "256x4"}
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    assert d["parity_ok"] is True
    assert d["delta_repair"]["ok"] is True and d["control_plane"]["ok"] is True
    rc = d["replica_compare"]
    assert set(rc) == {"0", "1", "64", "4096"} and all(v["exact"] for v in rc.values())
    assert all(v["sums_exact"] and v["sums_ms"] > 0 for v in rc.values())
    assert rc["0"]["n_diff"] == 0 and rc["1"]["n_diff"] == 1
    if "--no-cpu-baseline" not in extra:
        cb = d["cpu_baseline"]
        assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
        assert cb["one_thread"]["cores"] == 1 and cb["one_thread"]["value"] > 0
        assert set(cb["ops_gbs"]) == {"pack", "unpack", "verify", "checksum"}
