"""MX quantisation: Algorithm 2 (unbiased, stochastic rounding) and Algorithm 1.

Test infrastructure only (see the package docstring).

Algorithm 2 on one block V of k = 32 values:
  shared_exp = floor(log2 max_i |V_i|) - emax_elem        (emax_elem = 2 for E2M1)
  X = 2^shared_exp
  V_i <- (3/4) V_i ;  P_i = stochastic_round_to_FP4(V_i / X)
The 3/4 keeps every |V_i / X| below 6, the largest E2M1 value, so nothing is
clipped and the rounding stays unbiased (proof of Lemma 3.1).

Readings (the paper is silent on each):

* The scale X is stored as an E8M0 byte shared_exp + 127. floor(log2 0) is
  undefined and very small blocks would need shared_exp < -127; both clamp to
  the smallest E8M0 scale, byte 0. Clamping X upwards can never cause clipping.
* A block whose max |V_i| is not finite (inf or NaN) is outside the method's
  contract; it is flagged with the E8M0 NaN byte 0xFF and all-zero codes.
* (3/4) V_i / X is formed exactly and rounded to FP32 once.
* Stochastic rounding to the non-uniform E2M1 grid (Eq. 1 and the remark after
  it that the non-uniform case only rescales the noise): for a = |w| in the
  grid interval [f, c) with step D = c - f, let t = (a - f) / D in [0, 1).
  Eq. 1 on this interval rounds up iff t + delta >= 1/2 with delta uniform on
  [-1/2, 1/2). delta is drawn with 16 bits: delta = r / 2^16 - 1/2 for a 16-bit
  integer r, and t is taken at the same resolution, floor(t * 2^16). So the
  magnitude rounds up iff floor(t * 2^16) + r >= 2^16, which happens with
  probability floor(t * 2^16) / 2^16. The sign is kept, except that a zero
  magnitude always gets the code 0 (no negative zero).
* Cheaper-noise variant (a documented change of the rule above, selected
  explicitly, never the default): 8 bits, round up iff
  floor(t * 2^8) + r >= 2^8, probability floor(t * 2^8) / 2^8; its bias is at
  most 2^-8 of the grid step instead of 2^-16 (noise layout in ``philox``).
"""

import numpy as np

from .formats import E2M1_VALUES, E2M1_EMAX, E2M1_MAX, MX_BLOCK, E8M0_BIAS, E8M0_NAN
from .hadamard import rht_fp32
from .philox import sign_vector, noise16, noise8

SR_BITS = 16


def bf16_bits_to_fp32(bits):
    """bf16 bit patterns (uint16) to float32 values (exact: bf16 is the top half of FP32)."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def shared_exponent_byte(amax):
    """E8M0 byte of the shared exponent of Algorithm 2: floor(log2 amax) - emax_elem + 127, clamped to [0, 254].

    ``amax`` holds the per-block maxima |V|. Non-finite maxima give 0xFF.
    """
    amax = np.asarray(amax, dtype=np.float64)
    finite = np.isfinite(amax)
    positive = finite & (amax > 0)
    # frexp: amax = m * 2^e with m in [0.5, 1), so floor(log2 amax) = e - 1, exactly.
    _, e = np.frexp(np.where(positive, amax, 1.0))
    shared_exp = (e.astype(np.int64) - 1) - E2M1_EMAX
    byte = np.clip(shared_exp + E8M0_BIAS, 0, 254)
    byte = np.where(positive, byte, 0)
    return np.where(finite, byte, E8M0_NAN).astype(np.uint8)


def sr_e2m1(w, r16, bits=SR_BITS):
    """Stochastic rounding of float32 values |w| < 6 to E2M1 codes, with
    ``bits``-bit noise r16 (16, the method's rule; 8, the cheaper variant).

    Returns uint8 codes 0..15 (bit 3 = sign, bits 0..2 = index into the grid).
    """
    if bits not in (8, 16):
        raise ValueError("noise bits must be 16 or 8")
    w = np.asarray(w, dtype=np.float32)
    r16 = np.asarray(r16, dtype=np.int64)
    a = np.abs(w.astype(np.float64))
    if not np.all(a < E2M1_MAX):
        raise ValueError("stochastic rounding input outside the E2M1 range")
    idx = np.searchsorted(E2M1_VALUES, a, side="right") - 1       # f = E2M1_VALUES[idx] <= a
    f = E2M1_VALUES[idx]
    step = E2M1_VALUES[idx + 1] - f
    t = (a - f) / step                                            # exact in float64
    tq = np.floor(t * 2.0 ** bits).astype(np.int64)
    up = (tq + r16) >= 2 ** bits
    mag = idx + up.astype(np.int64)
    neg = np.signbit(w) & (mag != 0)
    return (mag | np.where(neg, 8, 0)).astype(np.uint8)


def _blocks(y):
    rows, cols = y.shape
    if cols % MX_BLOCK:
        raise ValueError("cols must be a multiple of 32")
    return y.reshape(rows, cols // MX_BLOCK, MX_BLOCK)


def mx_normalize(y):
    """Algorithm 2 up to the rounding: per 32-element block of the rows of
    float32 ``y``, the E8M0 scale byte and w = fl32((3/4) y / X).

    Returns (scales uint8 [rows, cols/32], w float32 [rows, cols]); blocks with a
    non-finite maximum get scale 0xFF and w = 0.
    """
    rows, cols = y.shape
    blocks = _blocks(y)
    amax = np.max(np.abs(blocks), axis=2)                          # float32, exact
    scales = shared_exponent_byte(amax)
    finite = scales != E8M0_NAN
    shared_exp = scales.astype(np.int64) - E8M0_BIAS
    # (3/4) V / X, exact in float64, then one rounding to FP32.
    factor = np.where(finite, 0.75 * np.ldexp(1.0, -shared_exp), 0.0)
    with np.errstate(invalid="ignore", over="ignore"):
        w = (blocks.astype(np.float64) * factor[:, :, None]).astype(np.float32)
    w = np.where(finite[:, :, None], w, np.float32(0.0)).reshape(rows, cols)
    return scales, w


def quantize_rht_sr(x_bits, g, seed, row_ids=None, rht=True, noise_bits=SR_BITS):
    """Blockwise RHT followed by Algorithm 2, on a logical [rows, cols] bf16 matrix.

    x_bits : uint16 bf16 bit patterns, the logical matrix (MX and RHT blocks run
             along each row). With ``row_ids`` it holds only those logical rows
             of a larger matrix; the noise is drawn for those row indices.
    g      : RHT block size (32 | g, g <= 256, power of two).
    seed   : 64-bit seed (hi32 selects the sign vector, all 64 bits the noise).
    rht    : False skips the transform (the "SR only" ablation of Table 2).
    noise_bits : 16 (the method) or 8 (the cheaper-noise variant; needs
             64 | cols).

    Returns (codes, scales): codes uint8 [rows, cols] one 4-bit code per element,
    scales uint8 [rows, cols/32] E8M0 bytes.
    """
    x = bf16_bits_to_fp32(x_bits)
    if x.ndim != 2:
        raise ValueError("expected a 2-D matrix")
    rows, cols = x.shape
    if g not in (32, 64, 128, 256):
        raise ValueError("g must be one of 32, 64, 128, 256")
    if cols % g:
        raise ValueError("g must divide cols")
    y = rht_fp32(x, sign_vector(seed, g)) if rht else x
    scales, w = mx_normalize(y)
    if row_ids is not None and len(row_ids) != rows:
        raise ValueError("row_ids must name every row of x_bits")
    if noise_bits == 8:
        codes = sr_e2m1(w, noise8(seed, rows, cols, row_ids), bits=8)
    else:
        codes = sr_e2m1(w, noise16(seed, rows, cols, row_ids))
    return codes, scales


def quantize_nr(x, rht_signs=None):
    """Algorithm 1 (OCP MX reference): shared scale as in Algorithm 2, no 3/4, nearest rounding.

    ``x`` is a float32 [rows, cols] matrix (optionally RHT'd first with
    ``rht_signs``). Ties round to the even grid index; values above 6 saturate.
    Returns (codes, scales, clipped) where ``clipped`` marks elements whose
    scaled magnitude exceeded 6 (Sec. 3.1: Algorithm 1 clips values in (6, 8)).
    """
    x = np.asarray(x, dtype=np.float32)
    y = rht_fp32(x, rht_signs) if rht_signs is not None else x
    rows, cols = y.shape
    blocks = _blocks(y)
    scales = shared_exponent_byte(np.max(np.abs(blocks), axis=2))
    if np.any(scales == E8M0_NAN):
        raise ValueError("non-finite input")
    v = blocks.astype(np.float64) * np.ldexp(1.0, -(scales.astype(np.int64) - E8M0_BIAS))[:, :, None]
    a = np.abs(v)
    clipped = a > E2M1_MAX
    a = np.minimum(a, E2M1_MAX)
    lo = np.clip(np.searchsorted(E2M1_VALUES, a, side="right") - 1, 0, 6)
    hi = lo + 1
    dlo = a - E2M1_VALUES[lo]
    dhi = E2M1_VALUES[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    mag = np.where(a >= E2M1_MAX, 7, np.where(pick_hi, hi, lo))
    neg = np.signbit(v) & (mag != 0)
    codes = (mag | np.where(neg, 8, 0)).astype(np.uint8)
    return codes.reshape(rows, cols), scales, clipped.reshape(rows, cols)


def pack_codes(codes):
    """[rows, cols] 4-bit codes -> [rows, cols/2] bytes, the even column in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 0::2] | (codes[:, 1::2] << np.uint8(4))).astype(np.uint8)


def unpack_codes(packed):
    """Inverse of ``pack_codes``."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows, half = packed.shape
    out = np.empty((rows, 2 * half), dtype=np.uint8)
    out[:, 0::2] = packed & np.uint8(0xF)
    out[:, 1::2] = packed >> np.uint8(4)
    return out
