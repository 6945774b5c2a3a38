"""GEMM parity across the whole E8M0 scale range, elementwise.

The normwise bound of the other GEMM tests (relative error 1e-5 over the whole
output) would hide one element that is off by a few percent, and their scale
bytes stay near 127. Here every output element is held to the rounding bound
of FP32 accumulation of exact products (proof of Lemma 3.1 writes the MXFP4
GEMM as a sum of exact FP4 x FP4 x 2^(sa + sb - 254) products):

  |C - C_ref| <= (K/32 + 32) 2^-24 (|deq A| |deq B|^T) + K 2^-126,

the first term covering one FP32 rounding per 64-element MFMA step and the
split-K reduction with a factor-2 margin, the second underflow below the
smallest normal FP32 value. The scale bytes span 0 .. 254 (each byte is
2^(byte - 127)) and 0xFF, the E8M0 NaN, which the quantiser writes for a block
holding an infinity or NaN: a product with such a block must be NaN, exactly
where the oracle's FP64 product is.
"""

import numpy as np
import pytest

import oracle
from oracle.mxquant import pack_codes
from workloads import matrix
from gpu_util import host, note, rel_err, to_dev, to_dev_u8, torch_gpu

pytestmark = pytest.mark.gpu


def _gemm_gpu(a, b, kernel=None):
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    m, n = a[0].shape[0], b[0].shape[0]
    c = torch.full((m, n), 12345.0, dtype=torch.float32, device="cuda")
    if kernel:
        mx.mx_profile_start()
    mx.mx_gemm_f4(to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])),
                  to_dev_u8(b[1]), c)
    if kernel:
        stats = mx.mx_profile_stop()
        assert kernel in stats, stats.keys()
    return host(c)


def _bound(a, b):
    k = a[0].shape[1]
    mag = np.abs(oracle.dequantize(*a)) @ np.abs(oracle.dequantize(*b)).T
    return (k / 32 + 32) * 2.0 ** -24 * mag + k * 2.0 ** -126


def _check_elementwise(got, a, b):
    ref = oracle.gemm_f64(*a, *b)
    nan_ref = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan_ref), (
        f"NaN positions differ: {int(np.isnan(got).sum())} on the GPU, {int(nan_ref.sum())} in the oracle")
    fin = ~nan_ref
    err = np.abs(got[fin].astype(np.float64) - ref[fin])
    bound = _bound(a, b)[fin]
    worst = np.argmax(err / bound)
    assert np.all(err <= bound), f"element error {err[worst]:.3g} above its bound {bound[worst]:.3g}"
    if fin.any():
        assert rel_err(got[fin], ref[fin]) <= 1e-5


def _codes(rng, rows, k):
    c = rng.integers(0, 16, size=(rows, k)).astype(np.uint8)
    c[c == 8] = 0
    return c


def _paired_scales(rng, m, n, k, spread, jitter):
    """A's scale bytes run over centre_kb +- jitter and B's over 254 - centre_kb +
    e_kb +- jitter: across the K blocks each operand's bytes cover 1 .. 254, while
    every product 2^(sa + sb - 254) stays within 2^(e_kb +- 2 jitter), e_kb drawn
    in [-spread, spread]."""
    kb = k // 32
    lo, hi = 1 + jitter, 254 - jitter
    centre = np.linspace(lo, hi, kb).round().astype(np.int64)
    rng.shuffle(centre)
    e = rng.integers(-spread, spread + 1, size=kb)
    sa = centre[None, :] + rng.integers(-jitter, jitter + 1, size=(m, kb))
    sb = np.clip(254 - centre + e, lo, hi)[None, :] + rng.integers(-jitter, jitter + 1, size=(n, kb))
    return sa.astype(np.uint8), sb.astype(np.uint8)


# One shape per GEMM kernel and a split-K one: (M, N, K, kernel).
SHAPES = [(300, 520, 1152, "gemm_128x128r"), (300, 520, 1056, "gemm_128x128"),
          (4096, 6144, 4096, "gemm_256x256"), (70, 1000, 6144, "gemm_128x128r")]


@pytest.mark.parametrize("m,n,k,kernel", SHAPES)
def test_scale_bytes_1_to_254_elementwise(m, n, k, kernel):
    """Each operand's scale bytes cover 1 .. 254; products stay near 2^0."""
    rng = np.random.default_rng(m + 3 * n + 7 * k)
    sa, sb = _paired_scales(rng, m, n, k, spread=0, jitter=4)
    assert sa.min() <= 5 and sa.max() >= 250 and sb.min() <= 5 and sb.max() >= 250
    a, b = (_codes(rng, m, k), sa), (_codes(rng, n, k), sb)
    note(f"gemm scales 1..254 M={m} N={n} K={k} {kernel}")
    _check_elementwise(_gemm_gpu(a, b, kernel), a, b)


@pytest.mark.parametrize("m,n,k,kernel", SHAPES)
def test_wide_product_range_elementwise(m, n, k, kernel):
    """Products of the K blocks range over 2^-100 .. 2^100: the FP32 sums are
    dominated by a few blocks and every element is held to its own bound."""
    rng = np.random.default_rng(5 + m + n + k)
    sa, sb = _paired_scales(rng, m, n, k, spread=100, jitter=3)
    a, b = (_codes(rng, m, k), sa), (_codes(rng, n, k), sb)
    note(f"gemm wide product range M={m} N={n} K={k} {kernel}")
    _check_elementwise(_gemm_gpu(a, b, kernel), a, b)


@pytest.mark.parametrize("m,n,k,kernel", SHAPES[:3])
def test_scale_byte_zero(m, n, k, kernel):
    """Byte 0 is 2^-127 (below the smallest normal FP32 value on its own): A's
    blocks with byte 0 meet B bytes of 200 .. 254, so their products are normal."""
    rng = np.random.default_rng(11 + m + k)
    kb = k // 32
    sa = rng.integers(120, 135, size=(m, kb)).astype(np.uint8)
    sb = rng.integers(120, 135, size=(n, kb)).astype(np.uint8)
    zero_cols = rng.choice(kb, size=max(1, kb // 4), replace=False)
    sa[:, zero_cols] = 0
    sb[:, zero_cols] = rng.integers(200, 255, size=(n, len(zero_cols)))
    a, b = (_codes(rng, m, k), sa), (_codes(rng, n, k), sb)
    note(f"gemm byte-0 scales M={m} N={n} K={k} {kernel}")
    _check_elementwise(_gemm_gpu(a, b, kernel), a, b)


@pytest.mark.parametrize("m,n,k,kernel", SHAPES)
def test_nan_scale_gives_nan(m, n, k, kernel):
    """A block with scale byte 0xFF (and, as the quantiser writes it, all-zero
    codes) makes its whole output row (A) or column (B) NaN; the rest is exact
    to the bound."""
    rng = np.random.default_rng(17 + m + n + k)
    kb = k // 32
    sa = rng.integers(118, 136, size=(m, kb)).astype(np.uint8)
    sb = rng.integers(118, 136, size=(n, kb)).astype(np.uint8)
    ca, cb = _codes(rng, m, k), _codes(rng, n, k)
    rows = rng.choice(m, size=min(m, 3), replace=False)
    cols = rng.choice(n, size=min(n, 5), replace=False)
    for r in rows:
        j = rng.integers(kb)
        sa[r, j] = 0xFF
        ca[r, 32 * j:32 * j + 32] = 0
    for c in cols:
        j = rng.integers(kb)
        sb[c, j] = 0xFF
        cb[c, 32 * j:32 * j + 32] = 0
    a, b = (ca, sa), (cb, sb)
    note(f"gemm NaN scales M={m} N={n} K={k} {kernel}")
    _check_elementwise(_gemm_gpu(a, b, kernel), a, b)


def test_quantiser_subnormal_blocks_through_the_gemm():
    """Quantiser output with byte-0 blocks (rows of subnormal bf16 inputs) times an
    operand with large scales, through the GPU quantiser and the GEMM."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    m, n, k, g = 256, 384, 1024, 64
    xa = matrix((m, k), seed=21)
    bits = xa.copy()
    # every 7th row: sign and the lowest mantissa bit only, i.e. +-2^-133 (the
    # smallest bf16 subnormal) or zero; a 64-block's transform is then at most
    # 2^-127, whose exponent field is 0, so its scale byte is 0
    bits[::7] = bits[::7] & 0x8001
    xb = matrix((n, k), seed=22, scale=2.0 ** 100)
    qa = oracle.quantize_rht_sr(bits, g, 0x77_0000_0001)
    qb = oracle.quantize_rht_sr(xb, g, 0x77_0000_0002)
    assert np.any(qa[1] == 0) and qb[1].min() > 200
    codes = torch.empty((m, k // 2), dtype=torch.uint8, device="cuda")
    scales = torch.empty((m, k // 32), dtype=torch.uint8, device="cuda")
    mx.mx_rht_sr_quantize(to_dev(bits), codes, scales, g, 0x77_0000_0001)
    assert np.array_equal(host(codes), pack_codes(qa[0])) and np.array_equal(host(scales), qa[1])
    note("gemm on quantiser output with byte-0 blocks")
    _check_elementwise(_gemm_gpu(qa, qb), qa, qb)


def test_linear_backward_nonfinite_inputs():
    """An infinity in dY and a NaN in x: dX, dW and db are NaN (or infinite)
    exactly where the oracle's are, and equal to it elsewhere."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fin, fout, g, seed = 256, 160, 128, 64, 0x1F_0000_0003
    dy = matrix((t, fout), 31, dist="t3", scale=1e-3)
    x = matrix((t, fin), 32)
    w = matrix((fout, fin), 33, scale=0.02)
    dy[17, 40] = 0x7F80          # +inf
    x[200, 99] = 0x7FC0          # NaN
    ref_dx, ref_dw, _ = oracle.linear_backward(dy, x, w, g, seed)
    ref_db = oracle.bias_grad(dy)
    dx = torch.empty((t, fin), dtype=torch.float32, device="cuda")
    dw = torch.empty((fout, fin), dtype=torch.float32, device="cuda")
    db = torch.empty((fout,), dtype=torch.float32, device="cuda")
    note("linear_backward_ex with inf in dY and NaN in x")
    mx.mx_linear_backward_ex(to_dev(dy), to_dev(x), to_dev(w), dx, dw, db, g, seed)
    for got, ref, name in ((host(dx), ref_dx, "dX"), (host(dw), ref_dw, "dW"), (host(db), ref_db, "db")):
        assert np.isnan(ref).any() or np.isinf(ref).any(), name
        assert np.array_equal(np.isnan(got), np.isnan(ref)), name
        assert np.array_equal(np.isinf(got), np.isinf(ref)), name
        fin_ = np.isfinite(ref)
        assert rel_err(got[fin_], ref[fin_]) <= 1e-5, name
