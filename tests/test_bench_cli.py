"""bench.py's command-line contract: one JSON line with the documented keys on an MI355X, and a
clear refusal of more than one GPU (runs without a GPU)."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")
KEYS = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
        "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"}
ROOF_KEYS = {"bound", "achieved", "peak", "unit", "frac", "traffic"}


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True,
                       timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr + r.stdout


def _run(*extra):
    r = subprocess.run([sys.executable, BENCH, "--steps", "3", "--warmup", "1", *extra],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    return json.loads(lines[0])


@pytest.mark.gpu
@pytest.mark.parametrize("workload", ["cfg2", "stats"])
def test_json_line(workload):
    out = _run("--workload", workload, "--cpu-seconds", "1")
    assert KEYS <= set(out)
    assert out["n_gpus"] == 1 and out["steps"] == 3 and out["warmup"] == 1
    assert out["value"] > 0 and out["ms_per_step"] > 0
    assert isinstance(out["config"]["workload"], str)
    roof = out["roofline"]
    assert ROOF_KEYS <= set(roof)
    assert 0 < roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"])
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["sample"]
    if workload == "cfg2":
        assert roof["frac_basis"].startswith("issued VALU lane-ops")
        assert "median" in roof["kernel_ms_statistic"] and roof["kernel_ms"] > 0


@pytest.mark.gpu
def test_default_line_carries_the_other_workloads():
    out = _run("--workload", "cfg3", "--cpu-seconds", "1", "--no-oracle-full")
    others = out["config"]["other_workloads"]
    assert set(others) == {"cfg0", "cfg1", "cfg2", "cfg4"}
    for name, o in others.items():
        assert o["scan_kernel_ms"] > 0 and 0 < o["frac"] < 1.5, name
        assert o["host_buffer_api"]["ms_per_call"] > 0
        assert o["ms_per_step"] > 0
    assert out["config"]["argmin"]["index"] >= 0
