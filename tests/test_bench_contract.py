"""The benchmark's output contract: one JSON line with the metric, the timing
fields, a roofline object for the dominant kernel and the CPU oracle's
throughput, and a refusal of more than one GPU (the path runs on one).  The
refusal runs on the CPU; the line itself needs the GPU (a short run of the
tiny workload)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True, timeout=300)
    assert res.returncode == 2
    assert "one GPU" in res.stdout + res.stderr
    assert res.stdout.strip() == "" or not res.stdout.strip().startswith("{")


@pytest.mark.gpu
def test_json_line_of_a_short_run():
    res = subprocess.run([sys.executable, "-u", BENCH, "--config", "tiny", "--steps", "3", "--warmup", "1",
                          "--cpu-budget", "0.5"], capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, res.stdout[-2000:]
    j = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in j, k
    assert j["n_gpus"] == 1 and j["steps"] == 3 and j["warmup"] == 1
    assert j["value"] > 0 and j["ms_per_step"] > 0 and j["higher_is_better"] is True
    assert j["config"]["workload"] == "tiny"
    r = j["roofline"]
    assert r["bound"] in ("hbm", "mfma", "alu")
    assert r["unit"] == ("GB/s" if r["bound"] == "hbm" else "TFLOP/s")
    assert r["achieved"] > 0 and r["peak"] > 0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-9
    assert "traffic" in r
    c = j["cpu_baseline"]
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1 and c["sample"]
