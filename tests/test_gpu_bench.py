"""bench.py end to end on the GPU with the tiny workload: one JSON line with
the contract's fields, a roofline object whose numbers follow from the
per-launch figures, the CPU oracle leg, and the timed output verified bit for
bit against the oracle's results."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("issue", ["engine", "launches"])
def test_bench_tiny_line(issue):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "2", "--warmup", "1",
           "--no-configs", "--cpu-seconds", "0.5", "--issue", issue]
    print(f"[bench tiny] {issue}", flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "verified"):
        assert key in line, key
    assert line["n_gpus"] == 1 and line["steps"] == 2 and line["warmup"] == 1 and line["value"] > 0
    assert line["config"]["issue"] == issue and line["config"]["workload"].startswith("tiny")
    rf = line["roofline"]
    assert rf["bound"] == "hbm" and rf["peak"] == 8000.0 and rf["unit"] == "GB/s"
    assert abs(rf["achieved"] - rf["bytes_per_launch"] / rf["avg_launch_us"] / 1e3) <= 0.01 * rf["achieved"] + 0.1
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert line["cpu_baseline"]["kind"] == "oracle" and line["cpu_baseline"]["value"] > 0
    assert line["verified"]["bit_exact"] is True
    other = "launches" if issue == "engine" else "engine"
    assert line[other]["value"] > 0
