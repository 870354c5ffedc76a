"""bench.py end to end on the GPU: a short run prints one JSON line with the keys
and units the measurement contract names (metric, value, roofline with its
algorithmic bytes and launch time, the CPU baseline of the oracle)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_short_bench_line():
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1",
           "--cpu-seconds", "1", "--no-configs", "--no-ceiling", "--layers", "4",
           "--variants", "bf16:weyl,e4m3:rtn"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline", "variants", "targets"):
        assert key in line, key
    assert line["n_gpus"] == 1 and line["steps"] == 3 and line["warmup"] == 1
    assert line["unit"] == "GB/s" and line["dtype"] == "f32" and line["data"] == "synthetic"
    assert line["config"]["workload"] == "hybrid_m2_stack" and "model" not in line["config"]
    roof = line["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["algorithmic_bytes_per_launch"] == 268435456 * 4
    # achieved = algorithmic bytes / average launch time; the line's value is the
    # same bytes per step over the step time, at most the kernel's own rate
    assert roof["achieved"] == pytest.approx(roof["algorithmic_bytes_per_launch"]
                                             / roof["avg_launch_us"] / 1e3, rel=1e-9)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-9)
    assert 0.2 < roof["frac"] < 1.0
    assert 0 < line["value"] <= roof["achieved"] * 1.001
    cpu = line["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0
    assert set(line["variants"]) == {"bf16:weyl", "e4m3:rtn"}
