"""GPU parity of the MXFP4 GEMM and of Algorithm 3 (mx_linear_backward).

GEMM outputs are compared with the oracle's FP64 product of the same
dequantised operands: normwise relative error at most 1e-5 (FP32 accumulation
of exact FP4 x FP4 x 2^k products; see the test module docstring of the CPU
oracle for the derivation of the bound). Algorithm 3 is compared the same way
after checking that its quantised operands are exactly the oracle's.
"""

import numpy as np
import pytest

import oracle
from oracle.mxquant import pack_codes, unpack_codes
from workloads import matrix, linear_inputs
from gpu_util import torch_gpu, to_dev, to_dev_u8, empty_u8, host, note, rel_err

pytestmark = pytest.mark.gpu

TOL = 1e-5


def _rand_mx(rng, rows, k, lo=118, hi=136):
    codes = rng.integers(0, 16, size=(rows, k)).astype(np.uint8)
    codes[codes == 8] = 0                      # canonical zero, as the quantiser produces
    scales = rng.integers(lo, hi, size=(rows, k // 32)).astype(np.uint8)
    return codes, scales


def _gemm_gpu(a, b):
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    m, n = a[0].shape[0], b[0].shape[0]
    c = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    mx.mx_gemm_f4(to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])),
                  to_dev_u8(b[1]), c)
    return host(c)


@pytest.mark.parametrize("m,n,k", [
    (1, 1, 32), (32, 32, 64), (100, 70, 96), (128, 128, 128), (256, 256, 256),
    (300, 520, 1056), (129, 257, 4096), (4096, 4096, 256), (4200, 4100, 160),
    (256, 256, 8192), (1024, 1024, 4096), (70, 1000, 6144),      # split along K
    (300, 520, 1152), (513, 257, 384), (1000, 24, 640), (2048, 1024, 3072),
])
def test_gemm_parity(m, n, k):
    rng = np.random.default_rng(m * 7 + n * 3 + k)
    a = _rand_mx(rng, m, k)
    b = _rand_mx(rng, n, k)
    note(f"gemm M={m} N={n} K={k}")
    got = _gemm_gpu(a, b)
    ref = oracle.gemm_f64(*a, *b)
    assert np.all(np.isfinite(got))
    assert rel_err(got, ref) <= TOL


@pytest.mark.parametrize("m,n,k,kernel", [(512, 384, 1024, "gemm_128x128r"), (4096, 5888, 4096, "gemm_128x128r"),
                                          (4096, 6144, 4096, "gemm_256x256"), (4096, 6144, 3968, "gemm_128x128r"),
                                          (512, 384, 1056, "gemm_128x128")])
def test_gemm_kernel_choice(m, n, k, kernel):
    """K % 128 == 0 runs an LDS-ring kernel (256 x 256 tiles when there are at least
    1.5 of them per CU, i.e. 384 on 256 CUs, and K is at least 4096, else
    128 x 128), other K the register-staged 128 x 128 one. 4096 x 5888 is 368
    256-tiles, 4096 x 6144 is 384."""
    import paper_2502_20586_amd as mx
    rng = np.random.default_rng(k)
    a = _rand_mx(rng, m, k)
    b = _rand_mx(rng, n, k)
    mx.mx_profile_start()
    got = _gemm_gpu(a, b)
    stats = mx.mx_profile_stop()
    assert kernel in stats and stats[kernel]["launches"] == 1
    assert rel_err(got, oracle.gemm_f64(*a, *b)) <= TOL


@pytest.mark.parametrize("m,n,k,kernel", [(300, 520, 1152, "gemm_128x128r"), (4096, 6144, 4096, "gemm_256x256"),
                                          (300, 520, 1056, "gemm_128x128")])
def test_gemm_output_aligned_to_one_element(m, n, k, kernel):
    """C only 4-byte aligned (16-byte aligned + 4), on each kernel: outputs are
    stored one element at a time, and the elements around C are left alone."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    rng = np.random.default_rng(m + n + k)
    a = _rand_mx(rng, m, k)
    b = _rand_mx(rng, n, k)
    buf = torch.full((m * n + 2,), -3.0, dtype=torch.float32, device="cuda")
    c = buf[1:1 + m * n].view(m, n)
    assert c.data_ptr() % 16 == 4
    note(f"gemm M={m} N={n} K={k} C at 16 B + 4")
    mx.mx_profile_start()
    mx.mx_gemm_f4(to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])), to_dev_u8(b[1]), c)
    stats = mx.mx_profile_stop()
    assert kernel in stats and stats[kernel]["launches"] == 1
    whole = host(buf)
    assert whole[0] == -3.0 and whole[-1] == -3.0
    assert rel_err(whole[1:1 + m * n].reshape(m, n), oracle.gemm_f64(*a, *b)) <= TOL


def test_gemm_on_quantised_data_and_determinism():
    rng = np.random.default_rng(1)
    xa = matrix((512, 768), seed=2, outlier_p=0.02, outlier_factor=100.0)
    xb = matrix((384, 768), seed=3, outlier_p=0.02, outlier_factor=100.0)
    qa = oracle.quantize_rht_sr(xa, 64, 11)
    qb = oracle.quantize_rht_sr(xb, 64, 12)
    g1 = _gemm_gpu(qa, qb)
    g2 = _gemm_gpu(qa, qb)
    assert np.array_equal(g1, g2)
    assert rel_err(g1, oracle.gemm_f64(*qa, *qb)) <= TOL


def test_split_k_gemm_is_deterministic():
    rng = np.random.default_rng(4)
    a = _rand_mx(rng, 200, 8192)
    b = _rand_mx(rng, 130, 8192)
    g1, g2 = _gemm_gpu(a, b), _gemm_gpu(a, b)
    assert np.array_equal(g1, g2)
    assert rel_err(g1, oracle.gemm_f64(*a, *b)) <= TOL


def test_release_workspace_between_gemms():
    """mx_release_workspace frees the stream's workspace in stream order: a GEMM
    enqueued before the release, one after it (which allocates again, here a
    split-K problem whose workspace also holds partial sums) and the release of
    a stream that holds none all give the oracle's results."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    rng = np.random.default_rng(11)
    a, b = _rand_mx(rng, 256, 8192), _rand_mx(rng, 384, 8192)
    assert mx.mx_gemm_f4_workspace_bytes(256, 384, 8192) > 256 * 8192 * 0.53
    ops = [to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])), to_dev_u8(b[1])]
    ref = oracle.gemm_f64(*a, *b)
    s = torch.cuda.Stream()
    outs = [torch.full((256, 384), float("nan"), device="cuda") for _ in range(2)]
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        mx.mx_gemm_f4(*ops, outs[0])
        mx.mx_release_workspace()
        mx.mx_release_workspace()                 # none left: still MX_OK
        mx.mx_gemm_f4(*ops, outs[1])
    torch.cuda.current_stream().wait_stream(s)
    s.synchronize()
    mx.mx_release_workspace(s)
    got = [host(c) for c in outs]
    assert np.array_equal(got[0], got[1])
    assert rel_err(got[0], ref) <= TOL
    fresh = torch.cuda.Stream()
    mx.mx_release_workspace(fresh)                # a stream the library never saw


def test_mfma_ceiling_is_plausible_and_above_the_gemm():
    """mx_measure_mfma_peak: FP4 MFMAs from registers run below the published
    10.1 PFLOP/s (the clock drops under full MFMA load) but well above what the
    GEMM kernel reaches, and at a clock under the nominal 2.4 GHz."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    note("mfma ceiling")
    tf, ghz = mx.mx_measure_mfma_peak(2000)
    assert 3000 < tf <= 10100 * 1.02, tf
    assert 0.8 < ghz < 2.5, ghz
    rng = np.random.default_rng(21)
    m = n = k = 8192
    a, b = _rand_mx(rng, m, k), _rand_mx(rng, n, k)
    ops = [to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), to_dev_u8(pack_codes(b[0])), to_dev_u8(b[1])]
    c = torch.empty((m, n), dtype=torch.float32, device="cuda")
    mx.mx_gemm_f4(*ops, c)
    mx.mx_profile_start()
    mx.mx_gemm_f4(*ops, c)
    st = mx.mx_profile_stop()["gemm_256x256"]
    gemm_tf = st["work"] / (st["total_ms"] * 1e-3) / 1e12
    assert gemm_tf < tf, (gemm_tf, tf)


def test_release_workspace_returns_memory():
    """After mx_release_workspace and a synchronisation the device has the
    workspace's memory back (the library's pool keeps no freed blocks)."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    m, n, k = 65536, 8192, 8192
    ws = mx.mx_gemm_f4_workspace_bytes(m, n, k)
    assert ws > 300e6
    a_codes = torch.zeros((m, k // 2), dtype=torch.uint8, device="cuda")
    a_scales = torch.full((m, k // 32), 127, dtype=torch.uint8, device="cuda")
    b_codes = torch.zeros((n, k // 2), dtype=torch.uint8, device="cuda")
    b_scales = torch.full((n, k // 32), 127, dtype=torch.uint8, device="cuda")
    c = torch.empty((m, n), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    note(f"workspace release: {ws / 1e6:.0f} MB")
    mx.mx_gemm_f4(a_codes, a_scales, b_codes, b_scales, c, stream=s)
    s.synchronize()
    assert torch.count_nonzero(c).item() == 0
    held = torch.cuda.mem_get_info()[0]
    mx.mx_release_workspace(s)
    s.synchronize()
    torch.cuda.synchronize()
    freed = torch.cuda.mem_get_info()[0] - held
    assert freed >= 0.9 * ws, (freed, ws)


def test_gemm_k_zero_and_empty():
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    c = torch.full((3, 5), 7.0, device="cuda")
    z = torch.empty((3, 0), dtype=torch.uint8, device="cuda")
    mx.mx_gemm_f4(z, z, torch.empty((5, 0), dtype=torch.uint8, device="cuda"),
                  torch.empty((5, 0), dtype=torch.uint8, device="cuda"), c)
    assert np.all(host(c) == 0.0)


def _backward_gpu(dy, x, w, g, seed):
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, out_f = dy.shape
    in_f = x.shape[1]
    dx = torch.full((t, in_f), float("nan"), dtype=torch.float32, device="cuda")
    dw = torch.full((out_f, in_f), float("nan"), dtype=torch.float32, device="cuda")
    mx.mx_linear_backward(to_dev(dy), to_dev(x), to_dev(w), dx, dw, g, seed)
    return host(dx), host(dw)


def test_linear_backward_tiny_config():
    dy, x, w = linear_inputs("tiny", "linear")
    note("linear_backward tiny T=256 in=out=256 g=64")
    dx, dw = _backward_gpu(dy, x, w, 64, 0)
    rdx, rdw, _ = oracle.linear_backward(dy, x, w, 64, 0)
    assert rel_err(dx, rdx) <= TOL and rel_err(dw, rdw) <= TOL


@pytest.mark.parametrize("t,fin,fout,g", [(64, 40, 64, 32), (128, 72, 256, 128), (256, 96, 512, 256),
                                          (192, 8, 64, 64)])
def test_linear_backward_shapes(t, fin, fout, g):
    dy = matrix((t, fout), seed=[t, 1], dist="t3", scale=1e-3, outlier_p=0.01, outlier_factor=100.0)
    x = matrix((t, fin), seed=[t, 2])
    w = matrix((fout, fin), seed=[t, 3], scale=0.02)
    seed = 0x5555_0000_0000_0007
    note(f"linear_backward T={t} in={fin} out={fout} g={g}")
    dx, dw = _backward_gpu(dy, x, w, g, seed)
    rdx, rdw, _ = oracle.linear_backward(dy, x, w, g, seed)
    assert rel_err(dx, rdx) <= TOL and rel_err(dw, rdw) <= TOL


def test_linear_backward_on_two_streams():
    """Calls on two streams with no synchronisation between them each use their own
    workspace; the larger call comes second on each stream, so both workspaces grow
    in stream order while earlier work may still be running."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    cases = [[(128, 64, 256, 64, 31), (512, 96, 1024, 64, 32)],
             [(256, 128, 128, 128, 33), (1024, 64, 512, 32, 34)]]
    jobs = []
    for st, per_stream in zip(streams, cases):
        for (t, fin, fout, g, seed) in per_stream:
            dy = matrix((t, fout), seed=[seed, 1], dist="t3", scale=1e-3)
            x = matrix((t, fin), seed=[seed, 2])
            w = matrix((fout, fin), seed=[seed, 3], scale=0.02)
            bufs = (to_dev(dy), to_dev(x), to_dev(w),
                    torch.full((t, fin), float("nan"), dtype=torch.float32, device="cuda"),
                    torch.full((fout, fin), float("nan"), dtype=torch.float32, device="cuda"))
            jobs.append((st, bufs, (dy, x, w, g, seed)))
    torch.cuda.synchronize()
    note("linear_backward on two streams")
    for st, b, (_, _, _, g, seed) in jobs:
        with torch.cuda.stream(st):
            mx.mx_linear_backward(*b, g, seed, stream=st)
    torch.cuda.synchronize()
    for _, b, (dy, x, w, g, seed) in jobs:
        rdx, rdw, _ = oracle.linear_backward(dy, x, w, g, seed)
        assert rel_err(host(b[3]), rdx) <= TOL and rel_err(host(b[4]), rdw) <= TOL


def test_linear_backward_equals_its_documented_composition():
    """dX / dW equal alpha * mx_gemm_f4 of the operands mx_rht_sr_quantize(_t)
    produce with seed ^ i, bit for bit."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fin, fout, g, seed = 256, 192, 128, 64, 0x1234_5678_9ABC_DEF0
    dy = matrix((t, fout), seed=21, dist="t3", scale=1e-3)
    x = matrix((t, fin), seed=22)
    w = matrix((fout, fin), seed=23, scale=0.02)
    dx, dw = _backward_gpu(dy, x, w, g, seed)
    ddy, dxx, dww = to_dev(dy), to_dev(x), to_dev(w)
    def q(src, rows, cols, i, transposed):
        c, s = empty_u8((rows, cols // 2)), empty_u8((rows, cols // 32))
        (mx.mx_rht_sr_quantize_t if transposed else mx.mx_rht_sr_quantize)(src, c, s, g, seed ^ i)
        return c, s
    q0 = q(ddy, t, fout, 0, False)
    q1 = q(dww, fin, fout, 1, True)
    q2 = q(ddy, fout, t, 2, True)
    q3 = q(dxx, fin, t, 3, True)
    alpha = np.float32(np.float32(16.0) / np.float32(9.0)) / np.float32(g)
    cx = torch.empty((t, fin), dtype=torch.float32, device="cuda")
    cw = torch.empty((fout, fin), dtype=torch.float32, device="cuda")
    mx.mx_gemm_f4(*q0, *q1, cx)
    mx.mx_gemm_f4(*q2, *q3, cw)
    assert np.array_equal(dx, host(cx) * alpha)
    assert np.array_equal(dw, host(cw) * alpha)


@pytest.mark.parametrize("name", ["qkv", "proj", "fc1", "fc2"])
def test_linear_backward_gpt345m_sampled(name):
    """GPT-345M layer shapes through mx_linear_backward as the benchmark calls
    it; sampled output rows are recomputed by the oracle (quantisation of every
    row of the B operand, sampled rows of the A operand)."""
    dy, x, w = linear_inputs("gpt345m", name)
    t, fout = dy.shape
    fin = x.shape[1]
    seed = 0x0345_0000_0000_0000
    note(f"linear_backward gpt345m {name} T={t} in={fin} out={fout}")
    dx, dw = _backward_gpu(dy, x, w, 64, seed)
    rng = np.random.default_rng(5)
    alpha = 16.0 / 9.0 / 64
    ids = np.unique(np.concatenate([[0, t - 1], rng.integers(0, t, 6)]))
    q0 = oracle.quantize_rht_sr(dy[ids], 64, seed ^ 0, row_ids=ids)
    q1 = oracle.quantize_rht_sr(np.ascontiguousarray(w.T), 64, seed ^ 1)
    assert rel_err(dx[ids], alpha * oracle.gemm_f64(*q0, *q1)) <= TOL
    ids = np.unique(np.concatenate([[0, fout - 1], rng.integers(0, fout, 6)]))
    dyt = np.ascontiguousarray(dy.T)
    q2 = oracle.quantize_rht_sr(dyt[ids], 64, seed ^ 2, row_ids=ids)
    q3 = oracle.quantize_rht_sr(np.ascontiguousarray(x.T), 64, seed ^ 3)
    assert rel_err(dw[ids], alpha * oracle.gemm_f64(*q2, *q3)) <= TOL


def test_kernel_tracing_counts_launches_and_work():
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fin, fout, g = 256, 128, 256, 64
    dy = to_dev(matrix((t, fout), seed=51))
    x = to_dev(matrix((t, fin), seed=52))
    w = to_dev(matrix((fout, fin), seed=53))
    dx = torch.empty((t, fin), dtype=torch.float32, device="cuda")
    dw = torch.empty((fout, fin), dtype=torch.float32, device="cuda")
    mx.mx_profile_start()
    for _ in range(3):
        mx.mx_linear_backward(dy, x, w, dx, dw, g, 9)
    stats = mx.mx_profile_stop()
    quant = [v for k, v in stats.items() if k.startswith("quant")]
    gemm = [v for k, v in stats.items() if k.startswith("gemm")]
    assert len(quant) == 1 and quant[0]["launches"] == 3 and not quant[0]["work_is_flops"]
    # Algorithmic bytes: each operand's codes and scales, and each input read
    # once (dY serves Q0 and Q2 in one pass at g = 64).
    assert quant[0]["work"] == 3 * ((t * fout + fin * fout + fin * t) * 2 + (2 * t * fout + fin * fout + fin * t) * (0.5 + 1 / 32))
    assert len(gemm) == 1 and gemm[0]["launches"] == 3 and gemm[0]["work_is_flops"]
    assert gemm[0]["work"] == 3 * 4 * t * fin * fout
    assert all(v["total_ms"] > 0 for v in stats.values())
    mx.mx_linear_backward(dy, x, w, dx, dw, g, 9)       # not traced once stopped
    assert mx.mx_profile_stop() == {}


def _check_backward_blocks(dy, x, w, g, seed, dx, dw, rng, n=8):
    """dX and dW on sampled row x column blocks against the oracle: the rows of
    both quantised operands that the block needs, quantised by the oracle
    (quantisation is row-local), multiplied in FP64."""
    t, fout = dy.shape
    fin = x.shape[1]
    alpha = 16.0 / 9.0 / g

    def pick(size):
        return np.unique(np.concatenate([[0, size - 1], rng.integers(0, size, n - 2)]))

    ri, ci, oi = pick(t), pick(fin), pick(fout)
    q0 = oracle.quantize_rht_sr(dy[ri], g, seed ^ 0, row_ids=ri)                          # Q(dY) rows
    q1 = oracle.quantize_rht_sr(np.ascontiguousarray(w[:, ci].T), g, seed ^ 1, row_ids=ci)  # Q(W^T) rows
    assert rel_err(dx[np.ix_(ri, ci)], alpha * oracle.gemm_f64(*q0, *q1)) <= TOL
    q2 = oracle.quantize_rht_sr(np.ascontiguousarray(dy[:, oi].T), g, seed ^ 2, row_ids=oi)  # Q(dY^T) rows
    q3 = oracle.quantize_rht_sr(np.ascontiguousarray(x[:, ci].T), g, seed ^ 3, row_ids=ci)   # Q(X^T) rows
    assert rel_err(dw[np.ix_(oi, ci)], alpha * oracle.gemm_f64(*q2, *q3)) <= TOL


@pytest.mark.parametrize("g", [32, 64, 128, 256])
def test_linear_backward_gpt1p3b_blocks(g):
    """GPT-1.3B fc1 (T = 8192, in = 2048, out = 8192) at full size for every g of
    the sweep; sampled blocks of dX and dW checked against the oracle."""
    dy, x, w = linear_inputs("gpt1.3b", "fc1")
    seed = 0x0130_0000_0000_0000 | g
    note(f"linear_backward gpt1.3b fc1 g={g}")
    dx, dw = _backward_gpu(dy, x, w, g, seed)
    assert np.all(np.isfinite(dx)) and np.all(np.isfinite(dw))
    _check_backward_blocks(dy, x, w, g, seed, dx, dw, np.random.default_rng(g))


@pytest.mark.parametrize("name", ["qkv", "proj", "fc1", "fc2"])
def test_linear_backward_gpt6p7b_blocks(name):
    """GPT-6.7B linears at full size (T = 16384, hidden 4096, dY with 0.5% of
    blocks x1000); sampled blocks of dX and dW checked against the oracle."""
    dy, x, w = linear_inputs("gpt6.7b", name)
    seed = 0x0670_0000_0000_0000
    note(f"linear_backward gpt6.7b {name} T={dy.shape[0]} in={x.shape[1]} out={dy.shape[1]}")
    dx, dw = _backward_gpu(dy, x, w, 64, seed)
    assert np.all(np.isfinite(dx)) and np.all(np.isfinite(dw))
    _check_backward_blocks(dy, x, w, 64, seed, dx, dw, np.random.default_rng(7))


def test_gemm_widest_output():
    """N = 2^24 - 1, the widest C the entry points take (a 32-row block of FP32
    C then spans just under 2^31 bytes of 32-bit buffer offsets), with ragged
    M = 40 (two row blocks, the second partial) and K = 128. B repeats a seeded
    block of 4096 rows; sampled columns, including the last ones, are checked
    against the oracle, and the canary past C is left alone."""
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    m, n, k = 40, (1 << 24) - 1, 128
    rng = np.random.default_rng(24)
    a = _rand_mx(rng, m, k)
    blk = _rand_mx(rng, 4096, k)
    reps = -(-n // 4096)
    b_codes = to_dev_u8(pack_codes(blk[0])).repeat(reps, 1)[:n].contiguous()
    b_scales = to_dev_u8(blk[1]).repeat(reps, 1)[:n].contiguous()
    buf = torch.full((m * n + 64,), -3.0, dtype=torch.float32, device="cuda")
    c = buf[:m * n].view(m, n)
    note(f"gemm M={m} N={n} K={k}")
    mx.mx_gemm_f4(to_dev_u8(pack_codes(a[0])), to_dev_u8(a[1]), b_codes, b_scales, c)
    cols = np.unique(np.concatenate([[0, 1, 4095, 4096, n // 2, n - 33, n - 2, n - 1], rng.integers(0, n, 8)]))
    got = host(c.index_select(1, torch.from_numpy(cols).to(c.device)))
    ref = oracle.gemm_f64(*a, blk[0][cols % 4096], blk[1][cols % 4096])
    assert rel_err(got, ref) <= TOL
    assert np.all(host(buf[m * n:]) == -3.0)
    del b_codes, b_scales, buf, c
    torch.cuda.empty_cache()
