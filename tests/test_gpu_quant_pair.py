"""GPU parity of mx_quantize_pair: both quantisations of one matrix (along its
rows and along its columns, Algorithm 3's two quantisations of dY) from one
pass over it, against the oracle's two separate quantisations, bit for bit.

Blocks of at most 64 take the one-pass path (each workgroup quantises the tile
it read in both directions); g = 128 and 256 run the two passes in one launch.
Shapes cover a single tile, ragged tiles in both directions (rows not a
multiple of 4 g, cols not a multiple of 64), every mode, three seeds each for
the pair, and canary bytes past both outputs.
"""

import numpy as np
import pytest

import oracle
from oracle.mxquant import bf16_bits_to_fp32, unpack_codes
from workloads import matrix
from gpu_util import torch_gpu, to_dev, empty_u8, host, note

pytestmark = pytest.mark.gpu

RHT_SR, SR, RHT_NR, NR, RHT_SR8 = 0, 1, 2, 3, 4
SEED_PAIRS = [(0, 2), (0x0123456789ABCDEF, 0x0123456789ABCDED), (0xFFFFFFFFFFFFFFFF, 7)]


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


def gpu_pair(bits, g, seed, seed_t, mode, canary_rows=2):
    torch_gpu()
    import paper_2502_20586_amd as mx
    rows, cols = bits.shape
    c = empty_u8((rows + canary_rows, cols // 2))
    s = empty_u8((rows + canary_rows, cols // 32))
    ct = empty_u8((cols + canary_rows, rows // 2))
    st = empty_u8((cols + canary_rows, rows // 32))
    mx.mx_quantize_pair(to_dev(bits), c[:rows], s[:rows], ct[:cols], st[:cols], g, seed, seed_t, mode)
    out = [host(t) for t in (c, s, ct, st)]
    for t in out:
        assert (t[-canary_rows:] == 0xA5).all(), "write past the end of an output"
    return (unpack_codes(out[0][:rows]), out[1][:rows]), (unpack_codes(out[2][:cols]), out[3][:cols])


def _check(bits, g, mode):
    for seed, seed_t in SEED_PAIRS:
        note(f"pair mode {mode} g={g} shape={bits.shape} seeds={seed:#x},{seed_t:#x}")
        (gc, gs), (gct, gst) = gpu_pair(bits, g, seed, seed_t, mode)
        oc, os_ = oracle_quant(bits, g, seed, mode)
        oct_, ost = oracle_quant(np.ascontiguousarray(bits.T), g, seed_t, mode)
        assert np.array_equal(gs, os_), f"row scales differ at {np.argwhere(gs != os_)[:5]}"
        assert np.array_equal(gc, oc), f"row codes differ at {np.argwhere(gc != oc)[:5]}"
        assert np.array_equal(gst, ost), f"column scales differ at {np.argwhere(gst != ost)[:5]}"
        assert np.array_equal(gct, oct_), f"column codes differ at {np.argwhere(gct != oct_)[:5]}"


@pytest.mark.parametrize("g", [32, 64, 128, 256])
def test_pair_rht_sr(g):
    # one tile; ragged in both directions; several row tiles and g-block groups
    for rmult, cols in ((1, g), (3, 5 * 32 if g <= 64 else g), (9, 4 * g)):
        rows = g * rmult
        cols = max(cols, g) // g * g
        bits = matrix((rows, cols), seed=[g, rows, cols], dist="t3", outlier_p=0.05, outlier_factor=100.0)
        _check(bits, g, RHT_SR)


@pytest.mark.parametrize("mode,g", [(SR, 64), (NR, 64), (RHT_NR, 32), (RHT_NR, 64), (RHT_SR8, 64),
                                    (RHT_SR8, 128)])
def test_pair_modes(mode, g):
    blk = g if mode in (RHT_SR, RHT_NR, RHT_SR8) else 32
    for rows, cols in ((blk, 2 * blk), (5 * blk, 3 * blk), (8 * blk, 96 if blk == 32 else 2 * blk)):
        bits = matrix((rows, cols), seed=[mode, g, rows, cols], outlier_p=0.05, outlier_factor=100.0)
        _check(bits, g, mode)


def test_pair_special_values():
    """Zero, subnormal, huge and non-finite blocks in both directions."""
    g = 64
    bits = matrix((256, 192), seed=91).copy()
    bits[3, :] = 0                       # zero row: zero blocks along the rows
    bits[:, 5] = 0x0001                  # a subnormal column
    bits[10, 64:128] = 0x7F7F            # huge block along a row
    bits[70, 7] = 0x7F80                 # +inf
    bits[200, 100] = 0x7FC1              # NaN
    for seed, seed_t in SEED_PAIRS[:2]:
        note(f"pair special values seeds={seed:#x},{seed_t:#x}")
        (gc, gs), (gct, gst) = gpu_pair(bits, g, seed, seed_t, RHT_SR)
        oc, os_ = oracle.quantize_rht_sr(bits, g, seed)
        oct_, ost = oracle.quantize_rht_sr(np.ascontiguousarray(bits.T), g, seed_t)
        assert np.array_equal(gs, os_) and np.array_equal(gc, oc)
        assert np.array_equal(gst, ost) and np.array_equal(gct, oct_)


def test_pair_gpt67b_shape_matches_separate_calls():
    """At a GPT-6.7B dY shape (16384 tokens x 4096), the pair equals the two
    mx_quantize calls byte for byte, and sampled rows of both equal the oracle."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, f, g = 16384, 4096, 64
    seed, seed_t = 0x6700000000000000, 0x6700000000000002
    gen = torch.Generator(device="cuda").manual_seed(67)
    x = torch.randn((t, f), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    c, s = empty_u8((t, f // 2)), empty_u8((t, f // 32))
    ct, st = empty_u8((f, t // 2)), empty_u8((f, t // 32))
    note("pair at 16384 x 4096 g=64")
    mx.mx_quantize_pair(x, c, s, ct, st, g, seed, seed_t, RHT_SR)
    c2, s2 = empty_u8((t, f // 2)), empty_u8((t, f // 32))
    ct2, st2 = empty_u8((f, t // 2)), empty_u8((f, t // 32))
    mx.mx_quantize(x, c2, s2, g, seed, RHT_SR, transposed=False)
    mx.mx_quantize(x, ct2, st2, g, seed_t, RHT_SR, transposed=True)
    torch.cuda.synchronize()
    for a, b in ((c, c2), (s, s2), (ct, ct2), (st, st2)):
        assert torch.equal(a, b)
    bits = x.view(torch.int16).cpu().numpy().view(np.uint16)
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, t - 1], rng.integers(0, t, 6)]))
    oc, os_ = oracle.quantize_rht_sr(bits[rows], g, seed, row_ids=rows)
    assert np.array_equal(unpack_codes(host(c)[rows]), oc) and np.array_equal(host(s)[rows], os_)
    cols = np.unique(np.concatenate([[0, f - 1], rng.integers(0, f, 6)]))
    xt = np.ascontiguousarray(bits[:, cols].T)
    oct_, ost = oracle.quantize_rht_sr(xt, g, seed_t, row_ids=cols)
    assert np.array_equal(unpack_codes(host(ct)[cols]), oct_) and np.array_equal(host(st)[cols], ost)
