"""The benchmark's output contract on the GPU: one short `bench.py` run (the
headline workload, few steps, the side measurements switched off) prints one
JSON line whose fields, units and roofline arithmetic are consistent and whose
parity check of the timed hot path passed."""
import json
import os
import subprocess
import sys

import pytest

from conftest import ROOT

pytestmark = pytest.mark.gpu


def _bench(*args, timeout=240):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT, capture_output=True,
                          text=True, timeout=timeout)


def test_bench_json_line():
    r = _bench("--steps", "20", "--warmup", "20", "--no-calib", "--no-gemm", "--no-table2",
               "--configs", "tiny_256x1152,shard_4608x1536", "--no-cpu-baseline")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 20 and d["warmup"] == 20
    assert d["unit"] == "GB/s" and d["higher_is_better"] is True and d["data"] == "synthetic"
    assert d["config"]["workload"] == "flux_4608x3072" and d["config"]["M"] == 4608 and d["config"]["d"] == 3072
    assert d["value"] > 0
    # value is the algorithmic bytes of one step over the measured time per step
    nbytes = 4608 * 3072 * (2 + 0.5 + 1 / 32)
    assert abs(d["value"] - nbytes / (d["ms_per_step"] * 1e-3) / 1e9) <= 1e-3 * d["value"] + 0.5
    # the stamps time exactly the K steps, inside the replay that the HIP events bracket
    ev = d["replay_events_us_per_launch"]["kroquant"] * (d["steps"] + d["warmup"])
    assert 0 < d["ms_per_step"] * 1e3 * d["steps"] <= ev * 1.001
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert rf["traffic"] is None or rf["traffic"] > nbytes * 0.99
    assert d["parity"]["hot_path"].startswith("ok"), d["parity"]
    assert d["parity"]["onthefly"].startswith("ok"), d["parity"]
    assert d["parity"]["exact_path"] == "bit-exact"
    # the quality side metric: a relative error in (0, 1) per method
    q = d["quantization_error"]
    assert all(0.0 < q[k] < 1.0 for k in ("kroquant", "smoothquant", "hadamard32", "mxfp4")), q
    # the single-launch ceiling: the best launch shape of the same traffic
    c = d["single_launch_ceiling"]
    assert c["us"] == min(c["sweep_us"].values()) and len(c["sweep_us"]) >= 10
    assert abs(d["hot_path_frac_of_ceiling"] - c["us"] / d["kernel_us"]) < 1e-3
    # the per-workload table: every kernel timed, its bandwidth the workload's bytes over its time
    for name, (M, dd) in (("tiny_256x1152", (256, 1152)), ("shard_4608x1536", (4608, 1536))):
        row = d["configs"][name]
        assert (row["M"], row["d"]) == (M, dd) and row["algorithmic_bytes"] == M * dd * (2 + 0.5 + 1 / 32)
        for k in ("kroquant_packed", "kroquant_onthefly", "kroquant_lu", "smoothquant", "hadamard32", "mxfp4",
                  "stream_floor"):
            gbs = row["algorithmic_bytes"] / row[k]["us"] * 1e-3
            assert row[k]["us"] > 0 and abs(row[k]["gbs"] - gbs) <= 1e-3 * gbs + 0.1

