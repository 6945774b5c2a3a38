"""Sylvester Hadamard matrix and the blockwise random Hadamard transform.

Test infrastructure only (see the package docstring).

Sec. 3.2 defines the RHT as x <- H S x with S a random sign vector and H the
Hadamard matrix given by the recursion that Sec. 3.2 writes down: H_n is built from four
copies of H_{n-1}, the lower-right one negated, starting from H_1 = [1].

Readings:

* Normalisation. The Hadamard recursion of Sec. 3.2 puts a factor 2^{-n/2} into a recursion whose
  H_{n-1} is already normalised, which cannot be what is meant; the intent is
  an orthogonal H (the paper notes H and diag(S) are orthogonal). The data
  path uses the +-1 Sylvester matrix, for which H H^T = g I, and the factor
  1/g this leaves in a product of two transformed operands is applied once,
  in the GEMM epilogue (see ``backward``).
* Block size. Algorithm 3 applies the transform in blocks of g elements along
  each operand's reduction dimension (the blockwise RHT of Sec. 3.2), with
  32 | g and g <= 256; one S of length g serves every block.
* Arithmetic. The paper only says the RHT runs in high precision. Here it is
  FP32 (IEEE round-to-nearest-even, no fused multiply-add, subnormals kept),
  and the transform is evaluated by the same recursion that defines H:
  H_n [a; b] = [H_{n-1} a + H_{n-1} b ; H_{n-1} a - H_{n-1} b], i.e. the two
  half-transforms are formed first and then added and subtracted. This fixes
  the order of every FP32 rounding.
"""

import numpy as np


def sylvester(g):
    """The g x g +-1 Sylvester Hadamard matrix (the Hadamard recursion of Sec. 3.2 without its scale factor), int64."""
    if g < 1 or (g & (g - 1)):
        raise ValueError("g must be a power of two")
    h = np.ones((1, 1), dtype=np.int64)
    while h.shape[0] < g:
        h = np.block([[h, h], [h, -h]])
    return h


def hadamard_fp32(x):
    """H_n x along the last axis of a float32 array, by the Hadamard recursion of Sec. 3.2.

    The length n of the last axis must be a power of two. Every add and subtract
    is a float32 operation, so each output is the FP32 value the recursion gives.
    """
    x = np.asarray(x)
    if x.dtype != np.float32:
        raise TypeError("hadamard_fp32 works on float32 data")
    n = x.shape[-1]
    if n == 1:
        return x.copy()
    half = n // 2
    a = hadamard_fp32(x[..., :half])
    b = hadamard_fp32(x[..., half:])
    return np.concatenate([a + b, a - b], axis=-1)


def rht_fp32(x, signs):
    """Blockwise RHT of the rows of a float32 [rows, cols] array: each g-block y = H_g (S o x).

    ``signs`` is the length-g vector S of +-1; g must divide cols. Multiplying by
    +-1 is exact, so only the Hadamard additions round.
    """
    x = np.asarray(x, dtype=np.float32)
    g = len(signs)
    rows, cols = x.shape
    if cols % g:
        raise ValueError("g must divide the number of columns")
    blocks = x.reshape(rows, cols // g, g) * np.asarray(signs, dtype=np.float32)
    return hadamard_fp32(blocks).reshape(rows, cols)
