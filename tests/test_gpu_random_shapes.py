"""GPU parity on seeded random shapes: ragged M, N (tails of every width inside a
tile and inside a pair of 32-column MFMA tiles), K of every residue mod 128
(ring and register-staged kernels), and mx_linear_backward_ex with every output
kind on random layer sizes. Same bars as the fixed-shape tests: GEMM outputs
within 1e-5 normwise of the oracle's FP64 product, bf16 dX within its rounding
bound, db within the summation bound.
"""

import numpy as np
import pytest

import oracle
from oracle.mxquant import pack_codes
from gpu_util import torch_gpu, to_dev_u8, host, note, rel_err
from test_gpu_integration import BF16, ACC, _check_bf16, _check_db, _inputs, _run_ex

pytestmark = pytest.mark.gpu

TOL = 1e-5


def _rand_mx(rng, rows, k):
    codes = rng.integers(0, 16, size=(rows, k)).astype(np.uint8)
    codes[codes == 8] = 0
    scales = rng.integers(112, 142, size=(rows, k // 32)).astype(np.uint8)
    return codes, scales


@pytest.mark.parametrize("case", range(16))
def test_gemm_random_shape(case):
    """Cases 0-11: M, N < 900, K a multiple of 128 (LDS-ring kernel) in even
    cases and of 32 in odd ones. Cases 12-15: M, N in [4900, 5300] and K >= 4096,
    at least 400 tiles of 256 x 256, so the 256 x 256 kernel runs with ragged
    edges."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    rng = np.random.default_rng(0x5EED_0000 + case)
    if case < 12:
        m, n = (int(v) for v in rng.integers(1, 900, size=2))
        k = (128 if case % 2 == 0 else 32) * int(rng.integers(1, 20 if case % 2 == 0 else 80))
    else:
        m, n = (int(v) for v in rng.integers(4900, 5300, size=2))
        k = 4096 + 128 * int(rng.integers(0, 8))
    a, b = _rand_mx(rng, m, k), _rand_mx(rng, n, k)
    note(f"gemm random case {case}: M={m} N={n} K={k}")
    c = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    mx.mx_profile_start()
    mx.mx_gemm_f4(to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])), to_dev_u8(b[1]), c)
    stats = mx.mx_profile_stop()
    if case >= 12:
        assert "gemm_256x256" in stats
    got = host(c)
    ref = oracle.gemm_f64(*a, *b)
    assert np.all(np.isfinite(got))
    assert rel_err(got, ref) <= TOL


@pytest.mark.parametrize("case", range(8))
def test_backward_ex_random_shape(case):
    """Random (T, in, out, g) with T and out multiples of g, in anything; each
    case runs one output kind (FP32, bf16 dX, accumulate, both), with db."""
    rng = np.random.default_rng(0xBAC0_0000 + case)
    g = int(rng.choice([32, 64, 128, 256]))
    t = g * int(rng.integers(1, 2048 // g + 1))
    fout = g * int(rng.integers(1, 1024 // g + 1))
    fin = int(rng.integers(1, 700))
    flags = [0, BF16, ACC, BF16 | ACC][case % 4]
    dy, x, w = _inputs(t, fin, fout, 1000 + case)
    seed = int(rng.integers(0, 2 ** 63))
    dw_main = db_main = None
    if flags & ACC:
        dw_main = rng.standard_normal((fout, fin)).astype(np.float32) * np.float32(1e-2)
        db_main = rng.standard_normal(fout).astype(np.float32)
    note(f"backward_ex random case {case}: T={t} in={fin} out={fout} g={g} flags={flags}")
    dx, dw, db = _run_ex(dy, x, w, g, seed, flags, True, dw_main=dw_main, db_main=db_main)
    rdx, rdw, _ = oracle.linear_backward(dy, x, w, g, seed)
    if flags & BF16:
        _check_bf16(dx, rdx)
    else:
        assert rel_err(dx, rdx) <= TOL
    if flags & ACC:
        assert rel_err(dw, dw_main.astype(np.float64) + rdw) <= TOL
        _check_db(db, dy, db_main)
    else:
        assert rel_err(dw, rdw) <= TOL
        _check_db(db, dy)
