"""GPU parity of mx_linear_backward_ex: bf16 dX, dW accumulation into an FP32
main gradient, and the bias gradient db = 1^T dY (Sec. 2.2), against the oracle.

Tolerances:
* FP32 dX / dW: normwise relative error at most 1e-5 against the oracle's FP64
  product of the same quantised operands (as for mx_linear_backward).
* bf16 dX: the FP32 result rounded to nearest bf16 (8 significant bits) is
  within 2^-8 |ref| of it, so every element must satisfy
  |dX - ref| <= 2^-8 |ref| + 1e-5 max |ref| (the second term covers the FP32
  accumulation error of elements near zero).
* Accumulated dW: main + dW, one FP32 rounding more than dW alone; normwise 1e-5
  against the oracle's main + dW in FP64.
* db: FP32 sums of T bf16 values in a fixed order of depth below T, so
  |db - exact| <= T 2^-24 sum_t |dY[t, j]| per column (the recursive-summation
  bound), and normwise relative error at most 1e-5.
"""

import numpy as np
import pytest

import oracle
from gpu_util import torch_gpu, to_dev, host, note, rel_err
from workloads import bf16_bits_to_float, linear_inputs, matrix

pytestmark = pytest.mark.gpu

TOL = 1e-5
BF16, ACC = 1, 2


def _inputs(t, fin, fout, key):
    dy = matrix((t, fout), seed=[key, 1], dist="t3", scale=1e-3, outlier_p=0.01, outlier_factor=100.0)
    x = matrix((t, fin), seed=[key, 2])
    w = matrix((fout, fin), seed=[key, 3], scale=0.02)
    return dy, x, w


def _run_ex(dy, x, w, g, seed, flags, with_db, mode=0, dw_main=None, db_main=None):
    """One mx_linear_backward_ex call; returns host copies (dX as bf16 bits when
    flags has BF16)."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fout = dy.shape
    fin = x.shape[1]
    if flags & BF16:
        dx = torch.full((t, fin), -1, dtype=torch.int16, device="cuda")      # 0xFFFF: a NaN canary
    else:
        dx = torch.full((t, fin), float("nan"), dtype=torch.float32, device="cuda")
    if dw_main is not None:
        dw = torch.from_numpy(np.ascontiguousarray(dw_main, dtype=np.float32)).cuda()
    else:
        dw = torch.full((fout, fin), float("nan"), dtype=torch.float32, device="cuda")
    db = None
    if with_db:
        db = (torch.from_numpy(np.ascontiguousarray(db_main, dtype=np.float32)).cuda() if db_main is not None
              else torch.full((fout,), float("nan"), dtype=torch.float32, device="cuda"))
    mx.mx_linear_backward_ex(to_dev(dy), to_dev(x), to_dev(w), dx, dw, db, g, seed, mode, flags)
    dxh = host(dx)
    if flags & BF16:
        dxh = dxh.view(np.uint16)
    return dxh, host(dw), (host(db) if with_db else None)


def _check_bf16(dx_bits, ref):
    got = bf16_bits_to_float(dx_bits).astype(np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    bound = 2.0 ** -8 * np.abs(ref) + 1e-5 * np.abs(ref).max()
    assert np.all(np.abs(got - ref) <= bound)


def _check_db(db, dy, main=None):
    exact = oracle.bias_grad(dy)
    if main is not None:
        exact = exact + np.asarray(main, dtype=np.float64)
    t = dy.shape[0]
    absum = np.abs(bf16_bits_to_float(dy).astype(np.float64)).sum(axis=0)
    if main is not None:
        absum = absum + np.abs(np.asarray(main, dtype=np.float64))
    assert np.all(np.abs(db.astype(np.float64) - exact) <= (t + 1) * 2.0 ** -24 * absum)
    assert rel_err(db, exact) <= TOL


# (T, in, out, g): ring-kernel shapes, a staged-kernel shape (K % 128 != 0), and
# shapes whose dW (first) or dX (second) GEMM is split along K, so the bf16 and
# accumulating stores also go through the split-K reduction.
SHAPES = [(256, 256, 256, 64), (96, 80, 96, 32), (4096, 128, 128, 64), (128, 128, 4096, 128),
          (512, 96, 1024, 256)]


@pytest.mark.parametrize("t,fin,fout,g", SHAPES)
@pytest.mark.parametrize("flags", [0, BF16, ACC, BF16 | ACC])
def test_backward_ex_against_oracle(t, fin, fout, g, flags):
    dy, x, w = _inputs(t, fin, fout, t + fin + fout + g)
    seed = 0x7777_0000_0000_0000 | (g << 4) | flags
    rng = np.random.default_rng(g + flags)
    dw_main = db_main = None
    if flags & ACC:
        dw_main = rng.standard_normal((fout, fin)).astype(np.float32) * np.float32(1e-2)
        db_main = rng.standard_normal(fout).astype(np.float32)
    note(f"backward_ex T={t} in={fin} out={fout} g={g} flags={flags}")
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


def test_backward_ex_without_options_is_mx_linear_backward():
    """No flags: dX and dW are bit for bit what mx_linear_backward writes, and the
    same with db requested (the column sums ride along in the dY^T pass)."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fin, fout, g, seed = 512, 192, 384, 64, 0xABCD_0000_1234_0000
    dy, x, w = _inputs(t, fin, fout, 5)
    dx0 = torch.empty((t, fin), dtype=torch.float32, device="cuda")
    dw0 = torch.empty((fout, fin), dtype=torch.float32, device="cuda")
    note("backward_ex vs mx_linear_backward")
    mx.mx_linear_backward(to_dev(dy), to_dev(x), to_dev(w), dx0, dw0, g, seed)
    for with_db in (False, True):
        dx, dw, _ = _run_ex(dy, x, w, g, seed, 0, with_db)
        assert np.array_equal(dx, host(dx0)) and np.array_equal(dw, host(dw0))


@pytest.mark.parametrize("mode", [1, 2, 3, 4])
def test_backward_ex_db_in_every_mode(mode):
    """Modes without the RHT sum dY in 32-element blocks, the RHT modes in g-blocks:
    db is the same column sum either way (within its bound)."""
    t, fin, fout = 1024, 64, 256
    dy, x, w = _inputs(t, fin, fout, 40 + mode)
    note(f"backward_ex db mode={mode}")
    _, _, db = _run_ex(dy, x, w, 128, 99, 0, True, mode=mode)
    _check_db(db, dy)


def test_backward_ex_db_is_deterministic_and_accumulates():
    """Two calls give the same db bit for bit; accumulating twice from zero gives
    db + db rounded once (exactly 2 db in FP32)."""
    t, fin, fout, g = 2048, 64, 1024, 64
    dy, x, w = _inputs(t, fin, fout, 51)
    note("backward_ex db determinism")
    _, _, db1 = _run_ex(dy, x, w, g, 3, 0, True)
    _, _, db2 = _run_ex(dy, x, w, g, 3, 0, True)
    assert np.array_equal(db1, db2)
    _, _, acc1 = _run_ex(dy, x, w, g, 3, ACC, True, dw_main=np.zeros((fout, fin)), db_main=np.zeros(fout))
    assert np.array_equal(acc1, db1)
    _, _, acc2 = _run_ex(dy, x, w, g, 3, ACC, True, dw_main=np.zeros((fout, fin)), db_main=acc1)
    assert np.array_equal(acc2, 2 * db1)


def test_backward_ex_degenerate_shapes():
    """in == 0: only db is computed. T == 0: dX has no elements, dW and db are
    cleared, or left as they are when accumulating. out == 0: dX is all zeros."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    dy, _, _ = _inputs(256, 8, 128, 61)
    e16 = lambda *s: torch.empty(s, dtype=torch.int16, device="cuda")
    e32 = lambda *s: torch.empty(s, dtype=torch.float32, device="cuda")
    note("backward_ex in=0 db only")
    db = torch.full((128,), float("nan"), device="cuda")
    mx.mx_linear_backward_ex(to_dev(dy), e16(256, 0), e16(128, 0), e32(256, 0), e32(128, 0), db, 64, 1)
    _check_db(host(db), dy)

    note("backward_ex T=0")
    dw = torch.full((128, 16), 3.0, device="cuda")
    db = torch.full((128,), 5.0, device="cuda")
    mx.mx_linear_backward_ex(e16(0, 128), e16(0, 16), to_dev(matrix((128, 16), 62)), e32(0, 16), dw, db, 64, 1,
                             0, ACC)
    assert np.all(host(dw) == 3.0) and np.all(host(db) == 5.0)
    mx.mx_linear_backward_ex(e16(0, 128), e16(0, 16), to_dev(matrix((128, 16), 62)), e32(0, 16), dw, db, 64, 1)
    assert np.all(host(dw) == 0.0) and np.all(host(db) == 0.0)

    note("backward_ex out=0 bf16 dX")
    dx = torch.full((64, 16), 7, dtype=torch.int16, device="cuda")
    mx.mx_linear_backward_ex(e16(64, 0), to_dev(matrix((64, 16), 63)), e16(0, 16), dx, e32(0, 16), e32(0),
                             64, 1, 0, BF16)
    assert np.all(host(dx) == 0)


def _all_options_sampled(dy, x, w, seed, kernel):
    """bf16 dX, dW accumulated into a main gradient and db, on the GEMM kernel
    named: db checked in full, dX and dW on sampled blocks."""
    import paper_2502_20586_amd as mx
    t, fout = dy.shape
    fin = x.shape[1]
    rng = np.random.default_rng(11)
    dw_main = rng.standard_normal((fout, fin)).astype(np.float32) * np.float32(1e-3)
    db_main = rng.standard_normal(fout).astype(np.float32) * np.float32(1e-2)
    mx.mx_profile_start()
    dx, dw, db = _run_ex(dy, x, w, 64, seed, BF16 | ACC, True, dw_main=dw_main, db_main=db_main)
    stats = mx.mx_profile_stop()
    assert kernel in stats and stats[kernel]["launches"] == 1
    _check_db(db, dy, db_main)
    assert not np.any((dx & 0x7F80) == 0x7F80)        # no Inf / NaN in the bf16 dX
    # Checked on the blocks: dX within the bf16 bound is within 2^-8 normwise;
    # dW - main is the new gradient up to one FP32 rounding of main + dW.
    ri = np.unique(np.concatenate([[0, t - 1], rng.integers(0, t, 6)]))
    ci = np.unique(np.concatenate([[0, fin - 1], rng.integers(0, fin, 6)]))
    q0 = oracle.quantize_rht_sr(dy[ri], 64, seed ^ 0, row_ids=ri)
    q1 = oracle.quantize_rht_sr(np.ascontiguousarray(w[:, ci].T), 64, seed ^ 1, row_ids=ci)
    _check_bf16(dx[np.ix_(ri, ci)], 16.0 / 9.0 / 64 * oracle.gemm_f64(*q0, *q1))
    dw_new = dw.astype(np.float64) - dw_main
    oi = np.unique(np.concatenate([[0, fout - 1], rng.integers(0, fout, 6)]))
    q2 = oracle.quantize_rht_sr(np.ascontiguousarray(dy[:, oi].T), 64, seed ^ 2, row_ids=oi)
    q3 = oracle.quantize_rht_sr(np.ascontiguousarray(x[:, ci].T), 64, seed ^ 3, row_ids=ci)
    ref = 16.0 / 9.0 / 64 * oracle.gemm_f64(*q2, *q3)
    assert rel_err(dw_new[np.ix_(oi, ci)], ref) <= TOL


@pytest.mark.parametrize("name", ["qkv", "fc1"])
def test_backward_ex_gpt345m_all_options(name):
    """GPT-345M linears at full size (128 x 128 tiles) with every option."""
    dy, x, w = linear_inputs("gpt345m", name)
    note(f"backward_ex gpt345m {name} all options")
    _all_options_sampled(dy, x, w, 0x0345_0000_0000_0001, "gemm_128x128r")


def test_backward_ex_all_options_on_256_tiles():
    """T = in = out = 4096: 512 tiles of 256 x 256, so the bf16 dX and the
    accumulated dW run on the 256 x 256 kernel."""
    dy, x, w = _inputs(4096, 4096, 4096, 40)
    note("backward_ex 4096^3 all options, 256 x 256 tiles")
    _all_options_sampled(dy, x, w, 0x0409_6000_0000_0001, "gemm_256x256")


def test_backward_ex_gpt6p7b_db():
    """GPT-6.7B QKV (T = 16384, out = 12288, dY with 0.5% of blocks x1000): 256
    block sums per column, db checked in full."""
    dy, x, w = linear_inputs("gpt6.7b", "qkv")
    note("backward_ex gpt6.7b qkv db")
    _, _, db = _run_ex(dy, x, w, 64, 0x0670_0000_0000_0001, 0, True)
    _check_db(db, dy)
