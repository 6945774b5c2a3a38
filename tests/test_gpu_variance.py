"""The variance of Algorithm 3's inner-product estimator through the HIP path,
against the oracle's closed form (the variance theorem of Sec. 3.2 and its
figure), and the flush-to-zero count of the quantiser (Sec. 4.1).

Samples A_i, B_i in R^b are the rows of two [n, b] matrices drawn as the
figure's caption says (N(0, 1) plus N(0, 5) outliers with probability p). For
each of S draws, mx_quantize quantises both with independent noise (seeds that
share the high word, i.e. one sign vector S, and differ in the low word),
mx_gemm_f4 multiplies them, and the diagonal of alpha C holds the n estimates
alpha Q(A_i)^T Q(B_i). Their sample variance over the draws, averaged over the
rows, must match the oracle's exact mean variance within 5 standard errors of
that average; the zero codes of A, averaged over the draws, must match the
oracle's expected count within 5 standard errors. Codes and scales being
bit-exact elsewhere, these checks pin the noise's distribution: independence
between elements and operands, and the rounding probabilities.
"""

import numpy as np
import pytest

import oracle
from gpu_util import note, to_dev, torch_gpu
from workloads import mixture_vectors

pytestmark = pytest.mark.gpu


def _draws(a_bits, b_bits, g, hi, draws, mode):
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    n, b = a_bits.shape
    da, db = to_dev(a_bits), to_dev(b_bits)
    ac = torch.empty((n, b // 2), dtype=torch.uint8, device="cuda")
    asc = torch.empty((n, b // 32), dtype=torch.uint8, device="cuda")
    bc = torch.empty_like(ac)
    bsc = torch.empty_like(asc)
    c = torch.empty((n, n), dtype=torch.float32, device="cuda")
    est = torch.empty((draws, n), dtype=torch.float64, device="cuda")
    zeros = torch.empty(draws, dtype=torch.float64, device="cuda")
    for d in range(draws):
        mx.mx_quantize(da, ac, asc, g, hi | (2 * d), mode)
        mx.mx_quantize(db, bc, bsc, g, hi | (2 * d + 1), mode)
        mx.mx_gemm_f4(ac, asc, bc, bsc, c)
        est[d] = torch.diagonal(c).double()
        zeros[d] = (((ac & 7) == 0).sum() + (((ac >> 4) & 7) == 0).sum()).double()
    torch.cuda.synchronize()
    return est.cpu().numpy(), zeros.cpu().numpy()


@pytest.mark.parametrize("b,rht", [(64, False), (64, True), (256, False), (256, True)])
def test_estimator_variance_and_zero_codes_match_the_oracle(b, rht):
    import paper_2502_20586_amd as mx
    n, p, draws = 512, 0.05, 200
    g = b
    hi = 0x0F16_0000_0000_0000 | (b << 32)
    a = mixture_vectors(n, b, p, [71, b, 0])
    bb = mixture_vectors(n, b, p, [71, b, 1])
    mode = mx.MX_MODE_RHT_SR if rht else mx.MX_MODE_SR
    note(f"variance b={b} rht={rht} draws={draws}")
    est, zeros = _draws(a, bb, g, hi, draws, mode)
    est *= oracle.estimator_alpha(g, rht)
    exact = oracle.inner_product_variance(a, bb, g, hi, hi | 1, rht)
    emp = est.var(axis=0, ddof=1)
    se = np.sqrt(np.sum(2.0 * exact ** 2 / (draws - 1))) / n
    assert abs(emp.mean() - exact.mean()) <= 5 * se, (emp.mean(), exact.mean(), se)
    # and the estimates are unbiased for the oracle's expected product
    ma = oracle.sr_moments(a, g, hi, rht)[0]
    mb = oracle.sr_moments(bb, g, hi | 1, rht)[0]
    mean_exact = oracle.estimator_alpha(g, rht) * np.sum(ma * mb, axis=1)
    z = (est.mean(axis=0) - mean_exact) / np.sqrt(exact / draws)
    assert np.abs(z).max() < 6 and abs(z.mean()) < 5 / np.sqrt(n)
    m0, v0 = oracle.expected_zero_codes(a, g, hi, rht)
    assert abs(zeros.mean() - m0) <= 5 * np.sqrt(v0 / draws) + 1e-9, (zeros.mean(), m0)
