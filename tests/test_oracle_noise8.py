"""Pins of the cheaper-noise variant of the rounding rule (8-bit dither):
round |w| up iff floor(t 2^8) + r >= 2^8, one Philox call per 16 elements.

* Exhaustive over the 256 noise values: P(up) = floor(t 2^8) / 2^8 exactly,
  and the bias of the rounded value is in (-2^-8 D, 0] (D the grid step).
* Its draws are the bytes of the same Philox outputs the 16-bit rule uses
  (Random123-pinned in test_oracle_philox), one chunk of 8 elements per
  call's first half and the chunk 32 columns further per its second half:
  every output byte serves exactly one element, so no two elements of a row
  share their noise.
* Unbiased over 10^4 seeds (Lemma 3.1) up to the 8-bit resolution.
"""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.formats import E2M1_VALUES
from oracle.gemm import dequantize
from oracle.hadamard import rht_fp32
from oracle.mxquant import bf16_bits_to_fp32, mx_normalize, quantize_rht_sr, sr_e2m1
from oracle.philox import noise16, noise8, sign_vector
from workloads import matrix


def test_exhaustive_8_bit_rounding_probability():
    rng = np.random.default_rng(5)
    w = np.concatenate([rng.uniform(-5.99, 5.99, 300), E2M1_VALUES[:7] + 1e-3, -E2M1_VALUES[1:7]]).astype(np.float32)
    for wv in w:
        codes = sr_e2m1(np.full(256, wv, np.float32), np.arange(256), bits=8)
        a = Fraction(abs(float(wv)))
        idx = int(np.searchsorted(E2M1_VALUES, float(a), side="right") - 1)
        f = Fraction(E2M1_VALUES[idx])
        c = Fraction(E2M1_VALUES[min(idx + 1, 7)])
        ups = int(np.sum((codes & 7) == idx + 1))
        t = (a - f) / (c - f) if c > f else Fraction(0)
        assert ups == int(t * 256)                 # floor(t 2^8) of the 256 values round up
        mean = f + (c - f) * Fraction(ups, 256)
        assert -(c - f) / 256 < mean - a <= 0


def test_8_bit_draws_are_the_bytes_of_the_16_bit_streams():
    seed, rows, cols = 0x1234_0000_5678, 3, 256
    n8 = noise8(seed, rows, cols)
    n16 = noise16(seed, rows, cols)
    for a in range(cols // 64):
        for b in range(4):
            base = 64 * a + 8 * b                  # the call's counter is this chunk's 16-bit counter
            words = [int(n16[0, base + 2 * i]) | (int(n16[0, base + 2 * i + 1]) << 16) for i in range(4)]
            for h in range(2):
                for e in range(8):
                    k = 8 * h + e
                    assert n8[0, base + 32 * h + e] == (words[k >> 2] >> (8 * (k & 3))) & 0xFF


def test_no_two_elements_share_their_noise():
    rows, cols = 4, 192
    draws = np.stack([noise8(0x42_0000_0000 | s, rows, cols) for s in range(48)])   # [seeds, rows, cols]
    for r in range(rows):
        cols_noise = draws[:, r, :].T                                                 # [cols, seeds]
        assert len({tuple(v) for v in cols_noise}) == cols
    counts = np.bincount(draws.ravel(), minlength=256)
    expect = draws.size / 256
    assert np.sum((counts - expect) ** 2 / expect) < 256 + 6 * np.sqrt(2 * 256)     # chi-square, 255 dof


@pytest.mark.slow
def test_8_bit_variant_is_unbiased_up_to_its_resolution():
    g = 64
    bits = matrix((2, 128), seed=11, outlier_p=0.25, outlier_factor=50.0)
    hi = 0x5EED0000_00000000
    y = rht_fp32(bf16_bits_to_fp32(bits), sign_vector(hi, g))
    scales, w = mx_normalize(y)
    xscale = oracle.e8m0_value(scales).repeat(32, axis=1)
    target = 0.75 * y.astype(np.float64)
    n = 10000
    acc = np.zeros(y.shape)
    for s in range(n):
        codes, sc = quantize_rht_sr(bits, g, hi | s, noise_bits=8)
        acc += dequantize(codes, sc)
    mean = acc / n
    a = np.abs(w.astype(np.float64))
    idx = np.searchsorted(E2M1_VALUES, a, side="right") - 1
    f, c = E2M1_VALUES[idx], E2M1_VALUES[np.minimum(idx + 1, 7)]
    sigma = np.sqrt((c - a) * (a - f) * xscale ** 2 / n)
    res = (c - f) * xscale / 256                     # the rule's bias bound
    dev = np.abs(mean - target)
    assert np.all(dev <= 5 * sigma + res + 1e-12 * np.abs(target))
    assert np.mean(dev <= 3 * sigma + res + 1e-12 * np.abs(target)) >= 0.99
