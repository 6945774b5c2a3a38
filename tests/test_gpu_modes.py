"""GPU parity of the quantiser's ablation modes (the rows of Table 2) and of
mx_linear_backward_mode.

* MX_MODE_SR: Algorithm 2 without the RHT; the oracle is quantize_rht_sr with
  rht=False (same noise layout).
* MX_MODE_RHT_NR / MX_MODE_NR: Algorithm 1 (no 3/4, round to nearest, ties to
  the even code, saturation at 6) after / without the RHT; the oracle is
  quantize_nr, which raises on non-finite input, so these modes are checked on
  finite data only.
* MX_MODE_RHT_SR8: the cheaper-noise variant (8-bit dither); the oracle is
  quantize_rht_sr with noise_bits=8.

Codes and scales must match bit for bit; GEMM outputs within normwise relative
error 1e-5 of the oracle's FP64 product with the mode's rescale.
"""

import numpy as np
import pytest

import oracle
from oracle.mxquant import bf16_bits_to_fp32, unpack_codes
from workloads import fp32_to_bf16_bits, matrix
from gpu_util import torch_gpu, to_dev, empty_u8, host, note, rel_err

pytestmark = pytest.mark.gpu

TOL = 1e-5
RHT_SR, SR, RHT_NR, NR, RHT_SR8 = 0, 1, 2, 3, 4
SEEDS = [0, 0x0123456789ABCDEF, 0xFFFFFFFFFFFFFFFF]


def oracle_quant(bits, g, seed, mode):
    if mode == RHT_SR:
        return oracle.quantize_rht_sr(bits, g, seed)
    if mode == SR:
        return oracle.quantize_rht_sr(bits, 32, seed, rht=False)
    if mode == RHT_SR8:
        return oracle.quantize_rht_sr(bits, g, seed, noise_bits=8)
    signs = oracle.sign_vector(seed, g) if mode == RHT_NR else None
    codes, scales, _ = oracle.quantize_nr(bf16_bits_to_fp32(bits), rht_signs=signs)
    return codes, scales


def gpu_quant(bits, g, seed, mode, transposed):
    torch_gpu()
    import paper_2502_20586_amd as mx
    rows, cols = bits.shape
    codes = empty_u8((rows, cols // 2))
    scales = empty_u8((rows, cols // 32))
    src = to_dev(np.ascontiguousarray(bits.T) if transposed else bits)
    mx.mx_quantize(src, codes, scales, g, seed, mode, transposed=transposed)
    return unpack_codes(host(codes)), host(scales)


def _check(bits, g, seed, mode, transposed):
    note(f"mode {mode} g={g} shape={bits.shape} seed={seed:#x} transposed={transposed}")
    gc, gs = gpu_quant(bits, g, seed, mode, transposed)
    oc, os_ = oracle_quant(bits, g, seed, mode)
    assert np.array_equal(gs, os_), f"scales differ at {np.argwhere(gs != os_)[:5]}"
    assert np.array_equal(gc, oc), f"codes differ at {np.argwhere(gc != oc)[:5]}"


@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("mode,g", [(SR, 64), (NR, 64), (RHT_NR, 32), (RHT_NR, 64), (RHT_NR, 128),
                                    (RHT_NR, 256), (RHT_SR8, 64), (RHT_SR8, 128), (RHT_SR8, 256)])
def test_modes_small_ragged(mode, g, transposed):
    # several quad groups and tiles, plus rows not a multiple of 16 or 64
    for rows, mult in ((1, 1), (37, 3), (130, 2), (64, 4)):
        cols = g * mult
        bits = matrix((rows, cols), seed=[g, rows, mode], outlier_p=0.05, outlier_factor=100.0)
        for seed in SEEDS:
            _check(bits, g, seed, mode, transposed)


def test_modes_ignore_g_without_rht():
    """Without the RHT the result does not depend on g."""
    bits = matrix((48, 256), seed=17)
    for mode in (SR, NR):
        ref = gpu_quant(bits, 64, 5, mode, False)
        for g in (32, 128, 256):
            got = gpu_quant(bits, g, 5, mode, False)
            assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])


def test_nearest_rounding_ties_and_saturation():
    """Algorithm 1 on values placed exactly on midpoints of the E2M1 grid (ties go
    to the even code) and on scaled values in (6, 8) (saturate to 6)."""
    amax_4 = [4.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5, -5.0,
              0.125, 0.375, 0.625, 1.0, 1.5, 2.25, 2.75, 3.25, 3.75, 4.5, 5.5, -4.5, -5.5, 0.0, -0.0, 6.0, -6.0]
    amax_7 = [7.0, 6.5, 7.5, -7.0, 6.25, -6.75, 5.75, 5.25] + [0.5 * i for i in range(24)]
    tiny = [2.0 ** -130 * (i + 1) for i in range(32)]             # subnormal block, E clamped at 0
    x = np.array([amax_4, amax_7, tiny, [-v for v in amax_7]], dtype=np.float32)
    bits = fp32_to_bf16_bits(x)
    assert np.array_equal(bf16_bits_to_fp32(bits), x)            # every value exact in bf16
    for transposed in (False, True):
        _check(bits, 64, 0, NR, transposed)


@pytest.mark.parametrize("mode", [RHT_SR, SR, RHT_NR, NR, RHT_SR8])
def test_linear_backward_modes(mode):
    """dX = alpha Q0 Q1^T and dW = alpha Q2 Q3^T with each operand quantised in
    `mode` (seed ^ i), alpha = (16/9 with SR) / (g with the RHT)."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    for t, fin, fout, g in ((256, 96, 512, 64), (128, 72, 256, 128), (512, 200, 384, 64 if mode == RHT_SR8 else 32)):
        dy = matrix((t, fout), seed=[t, mode, 1], dist="t3", scale=1e-3, outlier_p=0.01, outlier_factor=100.0)
        x = matrix((t, fin), seed=[t, mode, 2])
        w = matrix((fout, fin), seed=[t, mode, 3], scale=0.02)
        seed = 0x00AB_0000_0000_0000 | (mode << 8) | g
        note(f"linear_backward_mode mode={mode} T={t} in={fin} out={fout} g={g}")
        dx = torch.full((t, fin), float("nan"), dtype=torch.float32, device="cuda")
        dw = torch.full((fout, fin), float("nan"), dtype=torch.float32, device="cuda")
        mx.mx_linear_backward_mode(to_dev(dy), to_dev(x), to_dev(w), dx, dw, g, seed, mode)
        alpha = (16.0 / 9.0 if mode in (RHT_SR, SR, RHT_SR8) else 1.0) / (g if mode in (RHT_SR, RHT_NR, RHT_SR8) else 1)
        q0 = oracle_quant(dy, g, seed ^ 0, mode)
        q1 = oracle_quant(np.ascontiguousarray(w.T), g, seed ^ 1, mode)
        q2 = oracle_quant(np.ascontiguousarray(dy.T), g, seed ^ 2, mode)
        q3 = oracle_quant(np.ascontiguousarray(x.T), g, seed ^ 3, mode)
        assert rel_err(host(dx), alpha * oracle.gemm_f64(*q0, *q1)) <= TOL
        assert rel_err(host(dw), alpha * oracle.gemm_f64(*q2, *q3)) <= TOL


def test_default_entry_points_are_mode_rht_sr():
    """mx_rht_sr_quantize(_t) and mx_linear_backward equal their MX_MODE_RHT_SR forms."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    bits = matrix((64, 256), seed=23)
    for transposed in (False, True):
        a = gpu_quant(bits, 64, 9, RHT_SR, transposed)
        codes = empty_u8((64, 128))
        scales = empty_u8((64, 8))
        if transposed:
            mx.mx_rht_sr_quantize_t(to_dev(np.ascontiguousarray(bits.T)), codes, scales, 64, 9)
        else:
            mx.mx_rht_sr_quantize(to_dev(bits), codes, scales, 64, 9)
        assert np.array_equal(unpack_codes(host(codes)), a[0]) and np.array_equal(host(scales), a[1])
    dy, x, w = (to_dev(matrix(s, seed=i)) for i, s in enumerate([(128, 128), (128, 64), (128, 64)]))
    outs = []
    for fn in (lambda dx, dw: mx.mx_linear_backward(dy, x, w, dx, dw, 64, 3),
               lambda dx, dw: mx.mx_linear_backward_mode(dy, x, w, dx, dw, 64, 3, RHT_SR)):
        dx = torch.empty((128, 64), dtype=torch.float32, device="cuda")
        dw = torch.empty((128, 64), dtype=torch.float32, device="cuda")
        fn(dx, dw)
        outs.append((host(dx), host(dw)))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
