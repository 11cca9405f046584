"""The bench as the round-end measurement runs it: `bench.py --gpus 1 --steps 20 --warmup 5` in a
child process must print one JSON line on the headline workload (GAE 4096x256 fp32 with
truncation), with the roofline and CPU-baseline objects, and a timed region that fits inside the
child's own wall time."""
import json
import os
import subprocess
import sys
import time

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.gpu
def test_bench_driver_command():
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "1", "--steps", "20",
           "--warmup", "5", "--cpu-seconds", "2"]
    print("running:", " ".join(cmd), flush=True)
    t0 = time.perf_counter()
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300, cwd=ROOT)
    wall = time.perf_counter() - t0
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 20 and out["warmup"] == 5
    assert out["dtype"] == "f32" and out["unit"] == "GB/s" and out["higher_is_better"] is True
    assert out["timing"].startswith("eager")
    assert out["config"]["workload"].startswith("GAE 4096x256 fp32")
    assert out["config"]["N"] == 4096 and out["config"]["T"] == 256
    rf = out["roofline"]
    assert rf["bound"] == "hbm" and rf["peak"] == 8000.0 and rf["unit"] == "GB/s"
    assert rf["achieved"] > 0 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert "traffic" in rf
    cb = out["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    # the timed region (20 steps) lies inside the child's run
    assert out["ms_per_step"] * out["steps"] / 1e3 < wall
    # value is the algorithmic bytes over the timed time per step
    nbytes = out["config"]["algorithmic_bytes"]
    assert out["value"] == pytest.approx(nbytes / (out["ms_per_step"] * 1e-3) / 1e9, rel=1e-3)
