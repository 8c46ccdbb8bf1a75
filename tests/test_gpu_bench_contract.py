"""The benchmark's JSON line: a short run of `bench.py` (as a child process) prints one line
with the fields its contract names, the roofline of the dominant kernel consistent with its own
figures, and refuses more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=timeout, cwd=ROOT)


def test_short_run_prints_the_contract_line():
    print("\n[gpu case] bench.py --steps 4 --warmup 2 --no-cpu-baseline --no-extras", flush=True)
    r = _run("--steps", "4", "--warmup", "2", "--no-cpu-baseline", "--no-extras")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.strip().splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    line = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline"):
        assert key in line, key
    assert line["n_gpus"] == 1 and line["steps"] == 4 and line["warmup"] == 2
    assert line["value"] > 0 and line["higher_is_better"] is True
    assert abs(line["value"] * line["ms_per_step"] / 1e3 / line["config"]["global_batch"] - 1) < 0.3
    assert "workload" in line["config"]
    roof = line["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["bound"] in ("hbm", "mfma", "alu")
    assert roof["dominant"] in ("support", "active", "sweep")
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=2e-3, abs=2e-4)
    if roof["bound"] == "mfma":
        achieved = roof["algorithmic_flops_per_launch"] / (roof["avg_us"] * 1e-6) / 1e12
        assert roof["achieved"] == pytest.approx(achieved, rel=2e-3)
    us = roof["us_per_batch"]
    on_stream = [k for k in us if k != "sweep" or roof["sweep_stream"] == "the caller's"]
    assert roof["dominant"] == max(on_stream, key=us.get)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2", timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr)
