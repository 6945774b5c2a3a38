"""Pins of oracle.variance: the closed-form variance of the SR inner-product
estimator and the flush-to-zero probability, checked against the oracle's own
quantiser drawn over many seeds (a Monte-Carlo estimate that shares none of the
closed form's arithmetic) and against the single-element variance of Lemma 3.1
(Appendix C: Var = (c - a)(a - f) X^2 when t has at most 16 fractional bits)."""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.formats import E2M1_VALUES
from oracle.gemm import dequantize
from oracle.mxquant import quantize_rht_sr
from workloads import fp32_to_bf16_bits, mixture_vectors


def _mc(a, b, g, hi, draws, rht):
    """alpha Q(A_i)^T Q(B_i) for every row i and draw d: [draws, n]; zero-code counts of A per draw."""
    alpha = oracle.estimator_alpha(g, rht)
    out, zeros = [], []
    for d in range(draws):
        qa = quantize_rht_sr(a, g, hi | (2 * d), rht=rht)
        qb = quantize_rht_sr(b, g, hi | (2 * d + 1), rht=rht)
        out.append(alpha * np.sum(dequantize(*qa) * dequantize(*qb), axis=1))
        zeros.append(int(np.sum((qa[0] & 7) == 0)))
    return np.array(out), np.array(zeros)


@pytest.mark.slow
@pytest.mark.parametrize("rht", [False, True])
def test_closed_form_variance_matches_monte_carlo(rht):
    n, b, g, draws = 6, 64, 64, 4000
    hi = 0x7A11_0000_0000_0000
    a = mixture_vectors(n, b, 0.05, [70, 0])
    bb = mixture_vectors(n, b, 0.05, [70, 1])
    exact = oracle.inner_product_variance(a, bb, g, hi, hi | 1, rht)
    est, zeros = _mc(a, bb, g, hi, draws, rht)
    emp = est.var(axis=0, ddof=1)
    # sample variance of a near-normal sum: relative sd sqrt(2 / (draws - 1))
    rel = np.abs(emp / exact - 1.0)
    assert np.all(rel < 5 * np.sqrt(2.0 / (draws - 1))), (emp, exact)
    # the mean is A_i^T B_i's unbiased estimate (Lemma 3.1)
    assert np.all(np.abs(est.mean(axis=0) - np.sum(
        oracle.sr_moments(a, g, hi, rht)[0] * oracle.sr_moments(bb, g, hi | 1, rht)[0], axis=1)
        * oracle.estimator_alpha(g, rht)) <= 5 * np.sqrt(exact / draws))
    mean0, var0 = oracle.expected_zero_codes(a, g, hi, rht)
    assert abs(zeros.mean() - mean0) <= 5 * np.sqrt(var0 / draws) + 1e-9


def test_single_element_variance_is_lemma_3_1():
    """One nonzero element per 32-block: its w = (3/4) y / X takes values on a
    16-bit grid of its interval, so P(up) = t exactly and the variance of the
    dequantised element is (c - a)(a - f) X^2, exactly."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        idx = int(rng.integers(0, 7))
        f, c = Fraction(E2M1_VALUES[idx]), Fraction(E2M1_VALUES[idx + 1])
        t = Fraction(int(rng.integers(0, 1 << 16)), 1 << 16)
        w = f + (c - f) * t                      # |w| < 6, representable in FP32
        # a block whose max is 4 (scale byte 127: X = 1, w = (3/4) y) and element y = (4/3) w
        y = np.zeros((1, 32), dtype=np.float32)
        y[0, 0] = np.float32(4.0)
        y[0, 5] = np.float32(float(w * Fraction(4, 3)))
        if Fraction(float(y[0, 5])) * Fraction(3, 4) != w:
            continue                               # (4/3) w not exact in FP32: skip
        bits = fp32_to_bf16_bits(y)
        if bits[0, 5] << 16 != y.view(np.uint32)[0, 5]:
            continue                               # not a bf16 value: skip
        m, s2, pz = oracle.sr_moments(bits, 32, 0, rht=False)
        var = Fraction(float(s2[0, 5])) - Fraction(float(m[0, 5])) ** 2
        assert var == (c - w) * (w - f)
        assert pz[0, 5] == (float(1 - t) if f == 0 else 0.0)


def test_variance_is_zero_on_the_grid():
    # block maximum 8: X = 2, w = (3/4) y / 2 = 3 y / 8 lands on the grid values 3, 1.5, 0
    y = np.tile(np.array([8.0, -4.0, 0.0, 4.0] * 8, dtype=np.float32), (3, 1))
    bits = fp32_to_bf16_bits(y)
    m, s2, pz = oracle.sr_moments(bits, 32, 0, rht=False)
    assert np.all(s2 == m * m)
    assert np.array_equal(pz, (y == 0).astype(np.float64))    # zeros stay code 0, nothing else flushes
