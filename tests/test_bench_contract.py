"""bench.py's command-line contract: one JSON line with the metric, the
roofline and the CPU baseline on one GPU; any other GPU count is refused with
a message and exit status 2, before anything touches a GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    proc = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)
    assert proc.returncode == 2, proc.stderr[-2000:]
    line = json.loads(proc.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


@pytest.mark.gpu
def test_short_run_prints_the_contract_line():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    cmd = [sys.executable, "-u", BENCH, "--steps", "40", "--warmup", "5", "--rounds", "2",
           "--discard", "1", "--no-layer", "--no-batch", "--no-step14b", "--no-large",
           "--cpu-seconds", "1", "--floor-steps", "40"]
    print("[bench contract] " + " ".join(cmd[2:]), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert proc.returncode == 0, proc.stderr[-3000:]
    out = json.loads(proc.stdout.strip().splitlines()[-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline", "verified", "launch_floor"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 40 and out["warmup"] == 5
    assert out["unit"] == "GB/s" and out["value"] > 0 and out["higher_is_better"] is True
    assert "workload" in out["config"]
    r = out["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] == out["value"] and abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    c = out["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] >= 1 and c["value"] > 0 and c["sample"]
    # the time per step and the value describe the same launches
    us = out["ms_per_step"] * 1e3
    assert abs(out["config"]["served_bytes_per_gemv"] / (us * 1e-6) / 1e9 - out["value"]) \
        <= 0.01 * out["value"]
    # every arm was checked before it was timed (a failed check ends the run)
    assert out["verified"]["replicas_checked"] >= 1
