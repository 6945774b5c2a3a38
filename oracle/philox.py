"""Philox4x32-10 and the two random streams the method draws.

Test infrastructure only (see the package docstring).

The paper asks for two kinds of randomness and fixes neither generator:
a random sign vector S in {+-1}^g for the random Hadamard transform (Sec. 3.2:
one length-g vector is all the randomness the transform needs), and independent uniform dithering
noise for stochastic rounding (Eq. 1; Lemma 3.1 assumes independent noise).
Both are drawn here from Philox4x32-10, the counter-based generator of
Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3"
(SC'11), so that any element's randomness is a pure function of (seed, index).

Readings (the paper is silent on all of them):

* Seed split. A 64-bit seed; its high 32 bits alone select S, so operands that
  are multiplied together (and must share S) can use seeds that differ only in
  the low 32 bits, which then give them independent noise.
* Sign vector. key = (0, hi32(seed)); element j of S uses counter
  (j >> 7, 0, 0, 1), output word (j >> 5) & 3, bit j & 31; S_j = -1 iff that bit
  is 1. Counter word 3 = 1 keeps these draws apart from the noise draws.
* Noise. For element (r, c) of the logical [rows, cols] matrix being quantised,
  L = r * cols + c; key = (lo32(seed), hi32(seed)); counter = (lo32(L >> 3),
  hi32(L >> 3), 0, 0); output word (L >> 1) & 3; the element takes the low 16
  bits of that word if L is even, the high 16 bits if L is odd. So one
  generator call serves 8 consecutive elements of a row.
* 8-bit noise (the cheaper-noise variant, a documented change of the rounding
  rule, not the method's default): element (r, c) with c = 64 a + 32 h + 8 b + e
  (h in {0, 1}, b in 0..3, e in 0..7) takes byte k = 8 h + e, i.e. byte k & 3 of
  output word k >> 2, of Philox(counter = (lo32(P), hi32(P), 0, 0), key as
  above) with P = (r * cols + 64 a + 8 b) >> 3. So one generator call serves 16
  elements: the 8 at 64 a + 8 b and the 8 thirty-two columns further.
"""

import numpy as np

# Philox4x32 constants from the SC'11 paper: round multipliers and the Weyl
# sequence increments applied to the key between rounds.
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10_scalar(ctr, key, rounds=10):
    """One Philox4x32 block on Python ints: ctr is 4 words, key is 2 words."""
    c0, c1, c2, c3 = (int(v) & MASK32 for v in ctr)
    k0, k1 = (int(v) & MASK32 for v in key)
    for _ in range(rounds):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 32, p0 & MASK32
        hi1, lo1 = p1 >> 32, p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return c0, c1, c2, c3


def philox4x32_10(c0, c1, c2, c3, k0, k1, rounds=10):
    """Vectorised Philox4x32 over numpy arrays (broadcasting); returns 4 uint32 arrays."""
    u64 = np.uint64
    c0, c1, c2, c3 = (np.asarray(v, dtype=u64) & u64(MASK32) for v in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=u64) & u64(MASK32)
    k1 = np.asarray(k1, dtype=u64) & u64(MASK32)
    m32 = u64(MASK32)
    for _ in range(rounds):
        p0 = u64(PHILOX_M0) * c0
        p1 = u64(PHILOX_M1) * c2
        hi0, lo0 = p0 >> u64(32), p0 & m32
        hi1, lo1 = p1 >> u64(32), p1 & m32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        k0 = (k0 + u64(PHILOX_W0)) & m32
        k1 = (k1 + u64(PHILOX_W1)) & m32
    return tuple(v.astype(np.uint32) for v in (c0, c1, c2, c3))


def _split(seed):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & MASK32, seed >> 32


def sign_vector(seed, g):
    """Random sign vector S in {+1, -1}^g of the RHT (Sec. 3.2), as float64."""
    _, hi = _split(seed)
    j = np.arange(g, dtype=np.uint64)
    words = philox4x32_10(j >> np.uint64(7), 0, 0, 1, 0, hi)
    stacked = np.stack(words, axis=0)                       # [4, g]
    w = stacked[(j >> np.uint64(5)) & np.uint64(3), np.arange(g)]
    bit = (w.astype(np.uint64) >> (j & np.uint64(31))) & np.uint64(1)
    return np.where(bit == 1, -1.0, 1.0)


def noise16(seed, rows, cols, row_ids=None):
    """16-bit dithering noise for each element of a logical [rows, cols] matrix.

    ``row_ids`` (optional) selects which logical rows to draw, for checks on a
    sample of rows of a large matrix; the result then has len(row_ids) rows.
    Returns uint32 values in [0, 65536).
    """
    if cols % 8:
        raise ValueError("cols must be a multiple of 8")
    lo, hi = _split(seed)
    r = np.arange(rows, dtype=np.uint64) if row_ids is None else np.asarray(row_ids, dtype=np.uint64)
    groups = cols // 8
    q = r[:, None] * np.uint64(groups) + np.arange(groups, dtype=np.uint64)[None, :]   # L >> 3
    w = philox4x32_10(q & np.uint64(MASK32), q >> np.uint64(32), 0, 0, lo, hi)
    out = np.empty((len(r), groups, 8), dtype=np.uint32)
    for i in range(4):                      # word i serves elements 2i (low half) and 2i+1 (high half)
        out[:, :, 2 * i] = w[i] & np.uint32(0xFFFF)
        out[:, :, 2 * i + 1] = w[i] >> np.uint32(16)
    return out.reshape(len(r), cols)


def noise8(seed, rows, cols, row_ids=None):
    """8-bit dithering noise (the cheaper-noise variant) for each element of a
    logical [rows, cols] matrix, cols a multiple of 64; ``row_ids`` as for
    noise16. Returns uint32 values in [0, 256)."""
    if cols % 64:
        raise ValueError("cols must be a multiple of 64")
    lo, hi = _split(seed)
    r = np.arange(rows, dtype=np.uint64) if row_ids is None else np.asarray(row_ids, dtype=np.uint64)
    n64 = cols // 64
    a = np.arange(n64, dtype=np.uint64)[None, :, None]
    b = np.arange(4, dtype=np.uint64)[None, None, :]
    p = r[:, None, None] * np.uint64(cols // 8) + np.uint64(8) * a + b          # [rows, n64, 4]
    w = philox4x32_10(p & np.uint64(MASK32), p >> np.uint64(32), 0, 0, lo, hi)
    out = np.empty((len(r), n64, 2, 4, 8), dtype=np.uint32)                   # [row, a, h, b, e]
    for h in range(2):
        for e in range(8):
            k = 8 * h + e
            out[:, :, h, :, e] = (w[k >> 2] >> np.uint32(8 * (k & 3))) & np.uint32(0xFF)
    return out.reshape(len(r), cols)
