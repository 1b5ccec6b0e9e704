"""bench.py keeps its output contract: one JSON line with the metric, the
roofline of the dominant kernel and the oracle's CPU baseline; more than one
GPU is refused with a message (the library measures one GPU)."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


@pytest.mark.gpu
@pytest.mark.timeout(600)
def test_default_bench_line_has_roofline_and_cpu_baseline():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "1",
                        "--warmup", "1", "--cpu-seconds", "2"],
                       capture_output=True, text=True, timeout=580, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    out = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "config"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["value"] > 0
    roof = out["roofline"]
    assert roof["bound"] in ("mfma", "hbm", "alu") and 0 < roof["frac"] < 1
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert "peak_activation_gb_vs_U" in out
