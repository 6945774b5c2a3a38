"""Variance of the stochastic-rounding GEMM estimator and the flush-to-zero
probability, in closed form from the pinned rounding rule.

Test infrastructure only (see the package docstring).

Given the shared scales (deterministic: they depend on the block maxima, not on
the noise), Algorithm 2 rounds every element independently: |w| in the grid
interval [f, c] goes to c with probability P = floor(t 2^16) / 2^16,
t = (|w| - f) / (c - f), else to f (the rounding rule of ``mxquant``). So each
dequantised element q = sign(w) * {f or c} * X has

  E[q]   = sign(w) (f + P (c - f)) X,
  E[q^2] = ((1 - P) f^2 + P c^2) X^2,

and its variance is (c - a)(a - f) X^2 up to the 16-bit dither resolution
(Lemma 3.1 and its proof in Appendix C). Two operands quantised with
independent noise (different low seed words) give, for the inner product of a
row A_i with a row B_i over K elements,

  Var[Q(A_i)^T Q(B_i)] = sum_k E[qa_k^2] E[qb_k^2] - E[qa_k]^2 E[qb_k]^2,

exactly, because all 2K roundings are independent. The estimator of A_i^T B_i
that Algorithm 3 forms is alpha Q(A_i)^T Q(B_i) with alpha = 16/9 (undoing the
3/4 of both operands) and, with the RHT, a further 1/g (H H^T = g I for the
+-1 Hadamard); its variance is alpha^2 times the above. The sign vector S is
fixed by the high seed word: the variance is over the rounding noise for that
S, which is what the variance theorem of Sec. 3.2 bounds (with high
probability over S) and what its figure plots, averaged over samples of A, B.

An element is flushed to zero when its magnitude rounds to 0: |w| < 1/2 (f = 0)
and the rounding goes down, probability 1 - P; a zero |w| is always code 0.
Sec. 4.1 names this loss of small gradient values as the reason SR alone is
not enough.
"""

import numpy as np

from .formats import E2M1_VALUES, E8M0_BIAS
from .hadamard import rht_fp32
from .mxquant import SR_BITS, bf16_bits_to_fp32, mx_normalize
from .philox import sign_vector


def sr_moments(x_bits, g, seed, rht=True, noise_bits=SR_BITS):
    """Per element of a logical [rows, cols] bf16 matrix quantised as
    ``quantize_rht_sr(x_bits, g, seed, rht=rht)`` does: (E[q], E[q^2], P(code 0))
    over the rounding noise, in float64, with q the dequantised value (E2M1
    value times the block scale, no 3/4 or 1/g undone). Non-finite blocks are
    outside this function's contract."""
    x = bf16_bits_to_fp32(x_bits)
    y = rht_fp32(x, sign_vector(seed, g)) if rht else x
    scales, w = mx_normalize(y)
    if np.any(scales == 0xFF):
        raise ValueError("non-finite block")
    a = np.abs(w.astype(np.float64))
    idx = np.searchsorted(E2M1_VALUES, a, side="right") - 1
    f = E2M1_VALUES[idx]
    c = E2M1_VALUES[np.minimum(idx + 1, len(E2M1_VALUES) - 1)]
    t = np.where(c > f, (a - f) / np.where(c > f, c - f, 1.0), 0.0)
    p_up = np.floor(t * 2.0 ** noise_bits) / 2.0 ** noise_bits
    xs = np.ldexp(1.0, scales.astype(np.int64) - E8M0_BIAS).repeat(32, axis=1)
    sgn = np.where(np.signbit(w), -1.0, 1.0)
    mean = sgn * (f + p_up * (c - f)) * xs
    second = ((1.0 - p_up) * f * f + p_up * c * c) * xs * xs
    p_zero = np.where(f == 0.0, 1.0 - p_up, 0.0)
    return mean, second, p_zero


def estimator_alpha(g, rht):
    """alpha of Algorithm 3's estimator: 16/9, and 1/g with the +-1 RHT."""
    return 16.0 / 9.0 / (g if rht else 1)


def inner_product_variance(a_bits, b_bits, g, seed_a, seed_b, rht=True):
    """Var[alpha Q(A_i)^T Q(B_i)] for every row i of the logical [n, K]
    matrices A and B (bf16 bits), quantised with seeds seed_a and seed_b, which
    must share their high word (one sign vector) and differ in the low word
    (independent noise). Returns float64 [n]."""
    if (seed_a >> 32) != (seed_b >> 32) or seed_a == seed_b:
        raise ValueError("seeds must share hi32 and differ")
    ma, sa, _ = sr_moments(a_bits, g, seed_a, rht)
    mb, sb, _ = sr_moments(b_bits, g, seed_b, rht)
    var = np.sum(sa * sb - (ma * mb) ** 2, axis=1)
    return estimator_alpha(g, rht) ** 2 * var


def expected_zero_codes(x_bits, g, seed, rht=True):
    """Expected number of code-0 elements of quantize_rht_sr(x_bits, g, seed, rht=rht),
    and the variance of that count (a sum of independent Bernoulli variables)."""
    _, _, p = sr_moments(x_bits, g, seed, rht)
    return float(p.sum()), float((p * (1.0 - p)).sum())
