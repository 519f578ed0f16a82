"""bench.py end to end on the small float32 workload: one JSON line with the
fields the benchmark contract asks for, a roofline object for the similarity
kernel and the CPU reference timed beside it."""
import json
import os
import subprocess
import sys

import pytest

from tests.gpu_check import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line():
    say("bench.py --workload b16_n10k_d768_f32")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "b16_n10k_d768_f32",
                        "--steps", "5", "--warmup", "2", "--cpu-queries", "4", "--cpu-seconds", "0.5",
                        "--cpu-one-thread-queries", "1"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 5 and out["warmup"] == 2
    assert out["unit"] == "prompts/s" and out["higher_is_better"] is True and out["scaling"] == "weak"
    assert out["dtype"] == "f32" and out["config"]["workload"] == "b16_n10k_d768_f32"
    assert out["value"] > 0 and out["ms_per_step"] > 0
    # value is the whole job's throughput: B queries per step
    assert out["value"] == pytest.approx(16 / (out["ms_per_step"] * 1e-3), rel=0.25)
    rf = out["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert 0 < rf["frac"] < 1 and rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-3)
    cb = out["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
    assert cb["one_thread"]["cores"] == 1
