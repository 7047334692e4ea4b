"""The benchmark's JSON line on the GPU, on the small float32 workload: run as a child
process the way the benchmark is run, and checked for the fields its consumers read."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny_f32_T256_d256_V2048_P8",
                        "--steps", "3", "--warmup", "1", "--cpu-sample-rows", "256"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads([ln for ln in r.stdout.splitlines() if ln.startswith("{")][-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1 and d["dtype"] == "f32"
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["unit"] == "tokens/s"
    assert d["config"]["workload"] == "tiny_f32_T256_d256_V2048_P8"
    roof = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and 0 < roof["frac"] < 1
    assert roof["traffic"] is None  # the committed counter profile covers another workload
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert cpu["gflops"] > 0 and cpu["nproc"] >= 1 and "cpu_model" in cpu
    assert d["working_set_mib"]["allocated_during_steps"] == 0
    for part in ("fwd", "bwd", "fwd_bwd"):
        t = d["timing_ms"][part]
        assert 0 < t["min"] <= t["median"] <= t["max"] and t["min"] <= t["mean"] <= t["max"]
    assert d["bad_targets"] == 0
