"""Pins for the oracle's Algorithm 2 (scale, 3/4 pre-scale, stochastic rounding)
and Algorithm 1 (nearest rounding, used only as a check of the scale rule).

What fixes each part:
* shared exponent: the paper's bound m / 2^shared_exp in [4, 8) (Sec. 3.1), so
  after the 3/4 every block maximum lands in [3, 6) and nothing reaches 6
  (proof of Lemma 3.1); Algorithm 1 then clips roughly 3% of entries (Sec. 3.1);
* stochastic rounding: enumerating all 2^16 noise values gives the exact rounding
  distribution, whose mean is the input up to the 16-bit dither resolution and
  whose variance is (c - a)(a - f) (Appendix D);
* the whole quantiser is unbiased for 3/4 of the transformed input (Lemma 3.1):
  the empirical mean over 10^4 seeds lies within 3 sigma.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.formats import E2M1_VALUES, e2m1_value, e8m0_value
from oracle.hadamard import rht_fp32
from oracle.mxquant import (shared_exponent_byte, mx_normalize, sr_e2m1, quantize_rht_sr,
                            quantize_nr, pack_codes, unpack_codes, bf16_bits_to_fp32)
from oracle.gemm import dequantize
from oracle.philox import sign_vector
from workloads import fp32_to_bf16_bits, matrix

CONST = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def test_shared_exponent_byte_special_values():
    f32 = np.float32
    amax = np.array([1.0, 6.0, 7.999, 8.0, 0.0, 2.0 ** -126, 2.0 ** -140, np.inf, np.nan,
                     np.nextafter(f32(2.0), f32(0)), 3.0e38], dtype=np.float32)
    got = shared_exponent_byte(amax)
    # floor(log2 m) - 2 + 127
    expect = [125, 127, 127, 128, 0, 0, 0, 255, 255, 125, 252]
    assert list(got) == expect


def _adversarial_blocks():
    rng = np.random.default_rng(5)
    rows = []
    f32 = np.float32
    for p in range(-130, 127, 7):
        for top in (np.nextafter(f32(2.0 ** (p + 1)), f32(0)), f32(2.0 ** p), f32(1.5 * 2.0 ** p)):
            blk = (rng.uniform(-1, 1, 32) * float(top)).astype(np.float32)
            blk[rng.integers(32)] = top
            rows.append(blk)
    return np.stack(rows)


def test_no_clipping_and_block_max_in_3_to_6():
    bound = CONST["alg2_scaled_max_bound"]["value"]
    rng = np.random.default_rng(6)
    y = np.concatenate([
        _adversarial_blocks(),
        (rng.standard_normal((256, 32)) * np.exp(rng.uniform(-30, 30, (256, 1)))).astype(np.float32),
    ])
    scales, w = mx_normalize(y)
    assert np.all(np.abs(w) < bound)
    normal = (np.abs(y).max(axis=1) >= 2.0 ** -124)          # blocks whose scale is not clamped
    m = np.abs(w).max(axis=1)
    assert np.all(m[normal] >= 3.0) and np.all(m[normal] < 6.0)
    # the codes produced from these w are all on the grid and decode to within one step
    codes = sr_e2m1(w, np.zeros_like(w, dtype=np.uint32))
    assert np.all(np.abs(e2m1_value(codes)) <= np.abs(w) + 1e-30)   # zero noise rounds down


def test_zero_and_tiny_blocks():
    y = np.zeros((3, 32), np.float32)
    y[1, 3] = np.float32(2.0 ** -140)                      # subnormal
    y[2, :] = np.float32(-0.0)
    scales, w = mx_normalize(y)
    assert list(scales[:, 0]) == [0, 0, 0]
    assert w[1, 3] == np.float32(0.75 * 2.0 ** -13)          # 2^-140 * 0.75 * 2^127
    codes = sr_e2m1(w, np.zeros(w.shape, np.uint32))
    assert np.all(codes == 0)                                # -0.0 encodes as +0


def test_non_finite_block_is_flagged():
    x = np.zeros((2, 64), np.float32)
    x[0, 5] = np.inf
    x[1, 40] = np.nan
    bits = fp32_to_bf16_bits(x)
    bits[1, 40] = 0x7FC0
    codes, scales = quantize_rht_sr(bits, 64, 0, rht=False)
    assert scales[0, 0] == 0xFF and scales[0, 1] == 0
    assert scales[1, 1] == 0xFF and scales[1, 0] == 0
    assert np.all(codes == 0)


def _sr_exhaustive(wv):
    w = np.full(65536, wv, dtype=np.float32)
    codes = sr_e2m1(w, np.arange(65536, dtype=np.uint32))
    return e2m1_value(codes)


def _grid_neighbours(a):
    a = Fraction(a)
    grid = [Fraction(v) for v in E2M1_VALUES]
    f = max(v for v in grid if v <= a)
    c = min(v for v in grid if v > a) if a < 6 else None
    return f, c


def _sample_w():
    f32 = np.float32
    vals = [0.0, 0.25, 0.5, 0.75, 1.0, 1.25, 1.5, 2.5, 3.5, 5.0, 5.999, 1e-7, 2.0 ** -130]
    for g in E2M1_VALUES[1:]:
        vals += [float(np.nextafter(f32(g), f32(0))), float(np.nextafter(f32(g), f32(10)))]
    rng = np.random.default_rng(8)
    vals += list(rng.uniform(0, 6, 40))
    vals = [float(f32(v)) for v in vals if float(f32(v)) < 6.0]
    return vals + [-v for v in vals if v > 0]


def _halves(q):
    """E2M1 values are multiples of 1/2: return them as exact integers in units of 1/2."""
    h = np.rint(np.abs(q) * 2).astype(np.int64)
    assert np.array_equal(h / 2.0, np.abs(q))
    return h


def test_sr_exhaustive_distribution_mean_and_variance():
    """Over all 2^16 noise values: only the two neighbours f, c occur; the mean
    is |w| truncated to the 16-bit dither resolution (so it is within one 2^-16
    step below |w|, and exact when that step divides |w| - f); the variance is
    (c - mean)(mean - f), the closed form of Appendix D."""
    for wv in _sample_w():
        q = _sr_exhaustive(wv)
        a = abs(wv)
        f, c = _grid_neighbours(a)
        h = _halves(q)
        if Fraction(a) == f:
            assert np.all(h == 2 * f)                        # on the grid: deterministic
            continue
        assert set(np.unique(h).tolist()) <= {int(2 * f), int(2 * c)}
        mean = Fraction(int(h.sum()), 2 * 65536)
        assert 0 <= Fraction(a) - mean < (c - f) / 65536
        var = Fraction(int((h * h).sum()), 4 * 65536) - mean * mean
        assert var == (c - mean) * (mean - f)
        # sign is kept except for zero magnitudes
        assert np.all((np.sign(q) == np.sign(wv)) | (q == 0))


def test_sr_is_exact_mean_when_dither_resolution_divides():
    rng = np.random.default_rng(13)
    for k in rng.integers(1, 1 << 16, size=60):
        t = Fraction(int(k), 1 << 16)
        for f, c in zip(E2M1_VALUES[:-1], E2M1_VALUES[1:]):
            a = Fraction(f) + (Fraction(c) - Fraction(f)) * t
            assert float(np.float32(float(a))) == float(a)
            q = _sr_exhaustive(float(a))
            assert Fraction(int(_halves(q).sum()), 2 * 65536) == a


@pytest.mark.slow
@pytest.mark.parametrize("g", [64, 128])
def test_quantiser_is_unbiased_for_three_quarters_of_rht_input(g):
    """Lemma 3.1: E[deq(Q(x))] = (3/4) H S x. Empirical mean over 10^4 seeds
    (same sign vector, independent noise) within 3 sigma per element, sigma from
    the closed-form variance, plus the 16-bit dither-resolution bias. g = 128 is
    a case where the +-1 Hadamard differs from the orthonormal one by the
    irrational factor sqrt(128): the estimator is unbiased for H S x all the
    same."""
    bits = matrix((2, 128), seed=11, outlier_p=0.25, outlier_factor=50.0)
    hi = 0x5EED0000_00000000
    y = rht_fp32(bf16_bits_to_fp32(bits), sign_vector(hi, g))
    scales, w = mx_normalize(y)
    xscale = e8m0_value(scales).repeat(32, axis=1)
    target = 0.75 * y.astype(np.float64)
    n = 10000
    acc = np.zeros(y.shape)
    for s in range(n):
        codes, sc = quantize_rht_sr(bits, g, hi | s)
        assert np.array_equal(sc, scales)
        acc += dequantize(codes, sc)
    mean = acc / n
    a = np.abs(w.astype(np.float64))
    idx = np.searchsorted(E2M1_VALUES, a, side="right") - 1
    f, c = E2M1_VALUES[idx], E2M1_VALUES[np.minimum(idx + 1, 7)]
    var = (c - a) * (a - f) * xscale ** 2
    sigma = np.sqrt(var / n)
    tol = 3 * sigma + (c - f) * xscale / 65536 + 1e-12 * np.abs(target)
    dev = np.abs(mean - target)
    ongrid = var == 0
    assert np.all(dev[ongrid] <= (c - f)[ongrid] * xscale[ongrid] / 65536 + 1e-12 * np.abs(target[ongrid]))
    within = dev <= tol
    assert within.mean() >= 0.99                  # 3-sigma: about 0.3% expected outside
    assert np.all(dev <= 5 * sigma + (c - f) * xscale / 65536 + 1e-12 * np.abs(target))
    z2 = ((mean - target)[~ongrid] / sigma[~ongrid]) ** 2
    assert 0.75 < z2.mean() < 1.3                 # the variance formula is right too


def test_algorithm1_clips_about_three_percent():
    """Sec. 3.1: without the 3/4, Algorithm 1's scale maps block maxima into
    [4, 8) and roughly 3% of entries land above 6 and clip."""
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2048, 1024)).astype(np.float32)
    _, _, clipped = quantize_nr(x)
    frac = clipped.mean()
    approx = CONST["alg1_clip_fraction"]["approx"]
    assert approx / 3 < frac < approx * 4 / 3
    # with the RHT too (g = 64)
    _, _, clipped = quantize_nr(x, rht_signs=sign_vector(1 << 32, 64))
    assert approx / 3 < clipped.mean() < approx * 4 / 3


def test_algorithm1_nearest_rounding_values():
    x = np.array([[4.0, 0.24, 0.25, 0.26, 0.75, 1.25, 2.5, 3.5, 5.0, -2.9, 7.5] + [0.0] * 21],
                 dtype=np.float32)
    codes, scales, clipped = quantize_nr(x)
    assert scales[0, 0] == 127                    # floor(log2 7.5) - 2 = 0
    vals = e2m1_value(codes[0, :11])
    assert list(vals) == [4.0, 0.0, 0.0, 0.5, 1.0, 1.0, 2.0, 4.0, 4.0, -3.0, 6.0]
    assert clipped[0, 10] and clipped.sum() == 1


def test_pack_round_trip_and_nibble_order():
    rng = np.random.default_rng(10)
    codes = rng.integers(0, 16, size=(5, 64)).astype(np.uint8)
    packed = pack_codes(codes)
    assert packed.shape == (5, 32)
    assert np.all(packed[:, 0] == (codes[:, 0] | (codes[:, 1] << 4)))
    assert np.array_equal(unpack_codes(packed), codes)


def test_row_sampling_matches_full_quantise():
    bits = matrix((48, 128), seed=12, outlier_p=0.05, outlier_factor=100.0)
    codes, scales = quantize_rht_sr(bits, 64, 0xABCD_0000_0001)
    ids = np.array([3, 47, 0, 20])
    c2, s2 = quantize_rht_sr(bits[ids], 64, 0xABCD_0000_0001, row_ids=ids)
    assert np.array_equal(c2, codes[ids]) and np.array_equal(s2, scales[ids])


def test_quantiser_rejects_bad_arguments():
    bits = np.zeros((4, 64), np.uint16)
    with pytest.raises(ValueError):
        quantize_rht_sr(bits, 48, 0)
    with pytest.raises(ValueError):
        quantize_rht_sr(np.zeros((4, 96), np.uint16), 64, 0)
    with pytest.raises(ValueError):
        sr_e2m1(np.array([6.0], np.float32), np.array([0]))
