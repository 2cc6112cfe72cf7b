"""bench.py's output contract: one JSON line on stdout with the fields the
benchmark record needs (value, steps, roofline, cpu_baseline with its parity
sample), and a refusal of more than one GPU before anything touches a GPU."""
import json
import math
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True, timeout=60)
    assert res.returncode == 2
    assert res.stdout == ""
    assert "one GPU only" in res.stderr


@pytest.mark.gpu
def test_json_line_contract():
    """A short run on the heterogeneous batch (24 matrices, 6,144 tiles at
    T = 128): every field of the record is present and consistent."""
    steps, warmup = 5, 2
    cmd = [sys.executable, BENCH, "--workload", "hetero", "--budget", "0", "--T", "128", "--K", "5",
           "--steps", str(steps), "--warmup", str(warmup), "--cpu-seconds", "1"]
    print("[gpu-case] bench.py " + " ".join(cmd[2:]), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [ln for ln in res.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, res.stdout
    rec = json.loads(lines[0])

    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "step_ms", "cpu_baseline"):
        assert key in rec, key
    assert rec["n_gpus"] == 1 and rec["steps"] == steps and rec["warmup"] == warmup
    assert rec["unit"] == "TFLOP/s" and rec["higher_is_better"] is True
    assert rec["dtype"] == "f16" and rec["data"] == "synthetic" and rec["vs_baseline"] is None
    assert rec["config"]["tiles"] == 6144 and rec["config"]["launches_per_step"] == 1
    assert "workload" in rec["config"]
    # value is the work of a step over the wall-clock time of a step
    flops_step = rec["roofline"]["flops_per_launch"] * rec["config"]["launches_per_step"]
    assert math.isclose(rec["value"], flops_step / (rec["ms_per_step"] * 1e-3) / 1e12, rel_tol=2e-3)
    assert 0 < rec["value"] < 2500

    roof = rec["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 2500.0
    assert math.isclose(roof["frac"], roof["achieved"] / roof["peak"], rel_tol=1e-3)
    assert math.isclose(roof["achieved"], roof["flops_per_launch"] / (roof["mean_launch_ms"] * 1e-3) / 1e12,
                        rel_tol=2e-3)
    # the events of the timed region see no more than the wall clock does
    assert roof["mean_launch_ms"] <= rec["ms_per_step"] * 1.01
    assert roof["mfma_issued_fraction"] == 0.75  # the 128-tile kernel's symmetric step
    assert rec["step_ms"]["steps"] == steps and rec["step_ms"]["median"] > 0

    cpu = rec["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "TFLOP/s" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert isinstance(cpu["sample"], str) and cpu["sample"]
    par = cpu["parity"]
    assert par["tiles"] > 0 and par["bar"] == 2e-2
    assert 0 < par["p50"] <= par["max"] <= par["bar"]
