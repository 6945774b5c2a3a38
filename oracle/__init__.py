"""CPU oracle for the MXFP4 backward-pass hot path of "Training LLMs with MXFP4"
(Tseng, Yu, Park, AISTATS 2025).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call, link or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
path (no kernels, headers, tables or helpers); the only common dependency is the
seeded input generator in ``workloads/``, which holds none of the method's
arithmetic.

It is plain, slow and written to be checked against the paper by eye:

* ``philox``   -- Philox4x32-10 (Salmon et al., SC'11), the counter-based generator
                  that supplies the sign vector and the dithering noise.
* ``formats``  -- E2M1 element grid (Table 1; Sec. 2.5) and the E8M0 shared scale.
* ``hadamard`` -- Sylvester Hadamard matrix (the recursion of Sec. 3.2) and the blockwise random
                  Hadamard transform of Sec. 3.2.
* ``mxquant``  -- Algorithm 2 (unbiased MXFP4 quantisation with stochastic
                  rounding, Eq. 1) and Algorithm 1 (nearest rounding).
* ``gemm``     -- MXFP4_GEMM of Algorithm 3 as dequantise-then-FP64 product
                  (Appendix C, proof of Lemma 3.1).
* ``backward`` -- Algorithm 3, the linear-layer backward pass; the bias gradient
                  1^T dY (Sec. 2.2) and accumulation into main gradients.
* ``variance`` -- the variance of Algorithm 3's inner-product estimator and the
                  flush-to-zero probability, in closed form from the rounding
                  rule (the variance theorem of Sec. 3.2 and its figure; Sec. 4.1).

Every reading taken where the paper is silent or garbled is listed in the
docstring of the function that takes it.
"""

from .philox import philox4x32_10, philox4x32_10_scalar, sign_vector, noise16, noise8
from .formats import E2M1_VALUES, e2m1_value, e8m0_value
from .hadamard import sylvester, hadamard_fp32, rht_fp32
from .mxquant import (shared_exponent_byte, mx_normalize, sr_e2m1, quantize_rht_sr,
                      quantize_nr, pack_codes, unpack_codes)
from .gemm import dequantize, gemm_f64
from .backward import linear_backward, bias_grad, linear_backward_accumulate
from .variance import sr_moments, estimator_alpha, inner_product_variance, expected_zero_codes

__all__ = [
    "philox4x32_10", "philox4x32_10_scalar", "sign_vector", "noise16", "noise8",
    "E2M1_VALUES", "e2m1_value", "e8m0_value",
    "sylvester", "hadamard_fp32", "rht_fp32",
    "shared_exponent_byte", "mx_normalize", "sr_e2m1", "quantize_rht_sr", "quantize_nr",
    "pack_codes", "unpack_codes",
    "dequantize", "gemm_f64", "linear_backward", "bias_grad", "linear_backward_accumulate",
    "sr_moments", "estimator_alpha", "inner_product_variance", "expected_zero_codes",
]
