"""The benchmark's JSON line: one short run of bench.py (a child process)
carries every field of its contract, with the dominant kernel's roofline and
the oracle's CPU timing, and refuses more than one GPU."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, timeout=240):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_bench_line_fields():
    r = _run("--steps", "3", "--warmup", "1", "--cpu-seconds", "1", "--sets", "2")
    assert r.returncode == 0, r.stderr[-2000:]
    line = [l for l in r.stdout.splitlines() if l.startswith("{")][-1]
    d = json.loads(line)
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["value"] > 0 and d["higher_is_better"] is False and d["data"] == "synthetic"
    assert "workload" in d["config"] and "model" not in d["config"]
    roof = d["roofline"]
    assert roof["bound"] in ("hbm", "mfma", "alu") and roof["unit"] in ("GB/s", "TFLOP/s")
    assert roof["peak"] > 0 and 0 < roof["frac"] <= 1
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["sample"]
    for extra in ("tree_builder", "commit", "sample_accept"):
        assert d[extra]["us"] > 0, extra
    # every line (the smaller configurations too) names its own dominant
    # kernel; counter traffic is attached only to the workload it was taken on
    traffic_wl = json.load(open(os.path.join(ROOT, "profiles", "traffic.json"))).get("workload")
    for e in [json.loads(l) for l in r.stdout.splitlines() if l.startswith("{")]:
        roof = e["roofline"]
        assert roof["kernel"] in {k["kernel"] for k in e["kernels"].values()}, (e["config"]["workload"], roof)
        if not e["config"]["workload"].startswith(str(traffic_wl) + ":"):
            assert roof["traffic"] is None, e["config"]["workload"]


def test_bench_refuses_more_than_one_gpu():
    r = _run("--gpus", "2", timeout=60)
    assert r.returncode != 0 and "one GPU" in r.stderr
