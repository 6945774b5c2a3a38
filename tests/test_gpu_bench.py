"""bench.py end to end on the tiny block (one 256 x 256 linear, 256 tokens):
one JSON line on stdout with the contract's fields, a value that is the step's
GEMM FLOPs over its time, a roofline entry whose rate is its per-launch work
over its average launch time, and per-kernel times that fit in the step."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line_on_tiny_block():
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--config", "tiny", "--steps", "5", "--warmup", "2",
           "--no-cpu", "--no-baselines", "--no-variants", "--no-secondary", "--no-ceiling"]
    print("running:", " ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=110)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    res = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "kernels", "gemm_attainable"):
        assert key in res, key
    assert res["n_gpus"] == 1 and res["steps"] == 5 and res["warmup"] == 2
    assert res["config"]["workload"] == "tiny_block_backward"
    assert res["unit"] == "TFLOP/s" and res["higher_is_better"] is True
    assert res["config"]["gemm_flops_per_step"] == 4 * 256 * 256 * 256   # dX and dW: 2 T in out each
    assert res["value"] == pytest.approx(res["config"]["gemm_flops_per_step"] / (res["ms_per_step"] * 1e-3) / 1e12,
                                         rel=1e-9)
    roof = res["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-9)
    scale = 1e12 if roof["unit"] == "TFLOP/s" else 1e9
    assert roof["achieved"] == pytest.approx(roof["per_launch"] / (roof["avg_us"] * 1e-6) / scale, rel=1e-9)
    assert 0 < roof["frac"] < 1
    kernel_ms = sum(k["ms_per_step"] for k in res["kernels"].values())
    assert 0 < kernel_ms <= 1.2 * res["ms_per_step"]
