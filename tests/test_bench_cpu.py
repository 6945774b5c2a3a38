"""Host-side parts of bench.py that need no GPU: the one-GPU guard and the GEMM
attainable-time bound, checked against the roofline arithmetic of the
block backward (dX: M, N, K = T, in, out; dW: out, in, T; 2 M N K FLOPs; MXFP4
operands at 17/32 B per element, FP32 outputs written once)."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


class _Layer:
    def __init__(self, t, fin, fout):
        self.t, self.fin, self.fout = t, fin, fout


def _block(t, h, mlp):
    return [_Layer(t, h, 3 * h), _Layer(t, h, h), _Layer(t, h, mlp), _Layer(t, mlp, h)]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_attainable_gpt67b_is_the_mfma_time():
    """Every GEMM of the GPT-6.7B block has FLOP per byte above the ridge
    (10.1 PFLOP/s over 8 TB/s = 1262.5), so the bound is 13.19 TFLOP at the
    peak: 1306.35 us."""
    layers = _block(16384, 4096, 16384)
    a = bench.gemm_attainable(layers, 3.0)
    flops = sum(4 * L.t * L.fin * L.fout for L in layers)
    assert flops == 13194139533312
    assert a["mfma_bound_gemms"] == 8 and a["hbm_bound_gemms"] == 0
    assert a["us_per_step"] == pytest.approx(flops / 10.1e15 * 1e6, rel=1e-12)
    assert a["frac"] == pytest.approx(a["us_per_step"] / 3000.0, rel=1e-12)


def test_attainable_gpt345m_is_the_hbm_time():
    """At GPT-345M every GEMM is below the ridge: the bound is its bytes at
    8 TB/s. QKV's dX, for one: (4096 + 1024) x 3072 x 17/32 B of operands plus
    4096 x 1024 x 4 B of FP32 output."""
    layers = _block(4096, 1024, 4096)
    a = bench.gemm_attainable(layers, 1.0)
    assert a["mfma_bound_gemms"] == 0 and a["hbm_bound_gemms"] == 8
    total = 0.0
    for L in layers:
        for m, n, k in ((L.t, L.fin, L.fout), (L.fout, L.fin, L.t)):
            assert 2 * m * n * k / ((m + n) * k * 17 / 32 + 4 * m * n) < 10.1e15 / 8e12
            total += ((m + n) * k * 17 / 32 + 4 * m * n) / 8e12 * 1e6
    assert a["us_per_step"] == pytest.approx(total, rel=1e-12)
    assert a["us_per_step"] == pytest.approx(28.770304, rel=1e-9)
