"""bench.py end to end on the GPU, in a child process: one JSON line with the fields the
benchmark contract names, a roofline entry and the oracle's CPU baseline, on the small workload."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "20",
                        "--warmup", "3", "--cpu-budget", "1"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 20 and d["warmup"] == 3
    assert d["config"]["workload"] == "tiny" and d["dtype"] == "bf16" and d["data"] == "synthetic"
    assert d["config"]["row_pitch"] == d["config"]["hidden"] == 256  # no tuned pitch for 256-wide rows: packed
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert "traffic" in roof and "traffic_GBps" in roof
    assert roof["kernel"] in ("combine_kernel", "dispatch_bf16_kernel", "fused_bf16_kernel")
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0 and cpu["sample"]
    assert cpu["bit_identical_to_single_thread"] is True
    assert cpu["single_thread"]["cores"] == 1 and cpu["single_thread"]["value"] > 0
    assert roof["launches_sampled"] >= 20 and roof["launches_sampled_in_timed_region"] == 2
    assert d["device"]["arch"] == "gfx950"
