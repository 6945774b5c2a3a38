"""Host-side checks of the C ABI (no GPU needed).

* libmxfp4.so loads and exports every function include/mxfp4.h declares;
* argument validation rejects bad arguments with the documented status before
  any HIP call (so these run on a machine without a GPU);
* the workspace-size query matches the documented layout.
"""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mxfp4.h")

binding = pytest.importorskip("paper_2502_20586_amd.binding")


def _lib():
    try:
        return binding.load_library()
    except ImportError as e:
        pytest.skip(str(e))


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mx_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("mx_rht_sr_quantize", "mx_rht_sr_quantize_t", "mx_gemm_f4", "mx_linear_backward",
                     "mx_status_string"):
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = _lib()
    for name in _declared_functions():
        assert hasattr(lib, name), name
    # and nothing the header does not declare is exported with the mx_ prefix
    out = os.popen(f"nm -D --defined-only {binding.lib_path()}").read()
    exported = set(re.findall(r"\bT (mx_[a-z0-9_]+)\b", out))
    assert exported == set(_declared_functions())


def test_status_strings():
    lib = _lib()
    for code, name in binding._STATUS.items():
        assert lib.mx_status_string(code).decode().startswith(name)
    assert lib.mx_status_string(12345).decode() == "MX_ERR_UNKNOWN"


FAKE = 4096  # a non-null, 16-byte aligned address that validation never dereferences


@pytest.mark.parametrize("g,rows,cols,expect", [
    (48, 4, 96, -2), (16, 4, 32, -2), (512, 4, 512, -2),      # bad g
    (64, -1, 64, -3), (64, 4, -64, -3), (64, 4, 96, -3),       # bad shapes
    (32, 4, 48, -3),
])
def test_quantize_validation(g, rows, cols, expect):
    lib = _lib()
    for fn in (lib.mx_rht_sr_quantize, lib.mx_rht_sr_quantize_t):
        assert fn(FAKE, FAKE, FAKE, rows, cols, g, 0, None) == expect


def test_quantize_modes_validation():
    """mx_quantize: unknown modes are rejected; modes without the RHT ignore g and
    need only cols % 32 == 0."""
    lib = _lib()
    q = lib.mx_quantize
    for mode in (-1, 5, 99):
        assert q(FAKE, FAKE, FAKE, 4, 64, 64, 0, mode, 0, None) == -8
    # the 8-bit-noise variant pairs 32-element chunks: g = 32 is refused
    assert q(FAKE, FAKE, FAKE, 4, 64, 32, 0, binding.MX_MODE_RHT_SR8, 0, None) == -2
    assert lib.mx_linear_backward_mode(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 32, 0,
                                       binding.MX_MODE_RHT_SR8, None) == -2
    assert q(FAKE, FAKE, FAKE, 4, 64, 48, 0, binding.MX_MODE_RHT_NR, 0, None) == -2   # g checked with RHT
    assert q(FAKE, FAKE, FAKE, 4, 96, 64, 0, binding.MX_MODE_RHT_NR, 1, None) == -3   # cols % g
    for mode in (binding.MX_MODE_SR, binding.MX_MODE_NR):
        assert q(FAKE, FAKE, FAKE, 4, 48, 64, 0, mode, 0, None) == -3                  # cols % 32
        assert q(None, None, None, 0, 96, 48, 0, mode, 0, None) == 0                    # g ignored
        assert q(None, FAKE, FAKE, 4, 96, 48, 0, mode, 1, None) == -1


def test_quantize_pair_validation():
    """mx_quantize_pair: both directions' block rule (rows and cols multiples of the
    block), every output pointer and the 16-byte input alignment are checked first."""
    lib = _lib()
    f = lib.mx_quantize_pair
    RHT_SR, SR = binding.MX_MODE_RHT_SR, binding.MX_MODE_SR
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 128, 48, 0, 2, RHT_SR, None) == -2     # bad g
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 96, 128, 64, 0, 2, RHT_SR, None) == -3     # rows % g
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 128, 96, 64, 0, 2, RHT_SR, None) == -3     # cols % g
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 0, 2, 9, None) == -8           # bad mode
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 48, 64, 64, 0, 2, SR, None) == -3          # rows % 32
    for i in range(5):                                                                # each pointer
        args = [FAKE] * 5
        args[i] = None
        assert f(*args, 64, 128, 64, 0, 2, RHT_SR, None) == -1
    assert f(FAKE + 8, FAKE, FAKE, FAKE, FAKE, 64, 128, 64, 0, 2, RHT_SR, None) == -4  # in 16-byte aligned
    assert f(FAKE, FAKE, FAKE, FAKE + 2, FAKE, 64, 128, 64, 0, 2, RHT_SR, None) == -4
    assert f(None, None, None, None, None, 0, 128, 64, 0, 2, RHT_SR, None) == 0       # empty


def test_measure_mfma_peak_validation():
    """Arguments are checked before any device work: NULL outputs, then the round count."""
    import ctypes
    lib = _lib()
    a, b = ctypes.c_double(0.0), ctypes.c_double(0.0)
    assert lib.mx_measure_mfma_peak(2000, None, ctypes.byref(b)) == -1          # MX_ERR_NULL
    assert lib.mx_measure_mfma_peak(0, ctypes.byref(a), ctypes.byref(b)) == -3  # MX_ERR_SHAPE
    assert lib.mx_measure_mfma_peak((1 << 20) + 1, ctypes.byref(a), ctypes.byref(b)) == -3


def test_gemm_workspace_bytes():
    """mx_gemm_f4_workspace_bytes: 0 for invalid or empty sizes; for K % 128 == 0 at
    least the K-tiled copies of both operands (0.53125 byte per element, each part
    rounded up to 256 bytes); split-K partial sums on top when few tiles meet a long K."""
    lib = _lib()
    f = lib.mx_gemm_f4_workspace_bytes
    assert f(0, 64, 128) == 0 and f(64, 0, 128) == 0 and f(64, 64, 96 + 1) == 0 and f(-1, 64, 128) == 0
    assert f(64, 1 << 24, 128) == 0                                          # N limit
    up = lambda v: (v + 255) // 256 * 256
    for m, n, k in ((4096, 4096, 4096), (16384, 4096, 12288), (256, 384, 1024)):
        copies = up(m * k // 2) + up(m * k // 32) + up(n * k // 2) + up(n * k // 32)
        got = f(m, n, k)
        assert got >= copies, (m, n, k)
        assert got - copies in (0,) or (got - copies) % (m * n * 4) == 0, (m, n, k, got - copies)
    assert f(8192, 8192, 8192) == up(8192 * 4096) * 2 + up(8192 * 256) * 2   # many tiles: no split
    assert f(256, 256, 65536) > up(256 * 32768) * 2 + up(256 * 2048) * 2    # one tile, long K: split
    assert f(64, 64, 96) == 0                                                # K % 128 != 0: no copies


def test_linear_backward_modes_validation():
    lib = _lib()
    f = lib.mx_linear_backward_mode
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 64, 0, 7, None) == -8
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 48, 0, binding.MX_MODE_RHT_SR, None) == -2
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 96, 64, 64, 64, 0, binding.MX_MODE_RHT_NR, None) == -3
    # without the RHT only multiples of 32 are needed and g is ignored: these get as
    # far as the NULL output
    for mode in (binding.MX_MODE_SR, binding.MX_MODE_NR):
        assert f(FAKE, FAKE, FAKE, None, FAKE, 96, 64, 160, 48, 0, mode, None) == -1
        assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 80, 64, 64, 48, 0, mode, None) == -3


def test_quantize_null_and_alignment():
    lib = _lib()
    assert lib.mx_rht_sr_quantize(None, FAKE, FAKE, 4, 64, 64, 0, None) == -1
    assert lib.mx_rht_sr_quantize(FAKE, None, FAKE, 4, 64, 64, 0, None) == -1
    assert lib.mx_rht_sr_quantize(FAKE, FAKE, None, 4, 64, 64, 0, None) == -1
    assert lib.mx_rht_sr_quantize(FAKE + 2, FAKE, FAKE, 4, 64, 64, 0, None) == -4
    assert lib.mx_rht_sr_quantize(FAKE, FAKE + 2, FAKE, 4, 64, 64, 0, None) == -4
    # transposed read: 16-byte alignment only needed when rows % 8 == 0
    assert lib.mx_rht_sr_quantize_t(FAKE + 2, FAKE, FAKE, 8, 64, 64, 0, None) == -4
    assert lib.mx_rht_sr_quantize_t(FAKE + 1, FAKE, FAKE, 5, 64, 64, 0, None) == -4


def test_empty_problems_are_no_ops():
    lib = _lib()
    assert lib.mx_rht_sr_quantize(None, None, None, 0, 64, 64, 0, None) == 0
    assert lib.mx_rht_sr_quantize(None, None, None, 7, 0, 64, 0, None) == 0
    assert lib.mx_rht_sr_quantize_t(None, None, None, 0, 64, 64, 0, None) == 0
    assert lib.mx_gemm_f4(None, None, None, None, None, 0, 5, 64, None) == 0
    assert lib.mx_gemm_f4(None, None, None, None, None, 5, 0, 64, None) == 0
    assert lib.mx_linear_backward(None, None, None, None, None, 64, 0, 64, 64, 0, None) == 0


def test_gemm_validation():
    lib = _lib()
    assert lib.mx_gemm_f4(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 4, 48, None) == -3
    assert lib.mx_gemm_f4(FAKE, FAKE, FAKE, FAKE, FAKE, -1, 4, 64, None) == -3
    assert lib.mx_gemm_f4(FAKE, FAKE, FAKE, FAKE, None, 4, 4, 64, None) == -1
    assert lib.mx_gemm_f4(None, FAKE, FAKE, FAKE, FAKE, 4, 4, 64, None) == -1
    assert lib.mx_gemm_f4(FAKE + 4, FAKE, FAKE, FAKE, FAKE, 4, 4, 64, None) == -4
    assert lib.mx_gemm_f4(FAKE, FAKE, FAKE, FAKE, FAKE + 1, 4, 4, 64, None) == -4
    # the epilogue's 32-bit buffer offsets cover a 32-row block of C only for N < 2^24
    assert lib.mx_gemm_f4(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 1 << 24, 64, None) == -3


def test_linear_backward_validation():
    lib = _lib()
    f = lib.mx_linear_backward
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 40, 0, None) == -2
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 96, 64, 64, 64, 0, None) == -3    # g must divide T
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 96, 64, 0, None) == -3    # g must divide out
    assert f(FAKE, FAKE, FAKE, None, FAKE, 64, 64, 64, 64, 0, None) == -1
    assert f(FAKE, None, FAKE, FAKE, FAKE, 64, 64, 64, 64, 0, None) == -1
    assert f(FAKE + 8, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 64, 0, None) == -4
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 64, 1 << 24, 64, 64, 0, None) == -3  # in_features is the GEMMs' N


def test_workspace_bytes_layout():
    """Scratch holds the four quantised operands (codes + scales, 256-byte
    aligned parts) and, when a GEMM is split along K, its partial sums."""
    lib = _lib()
    def up(v):
        return (v + 255) // 256 * 256
    for t, fin, fout in ((4096, 1024, 3072), (256, 256, 256), (64, 40, 64)):
        quant = 0
        for n in (t * fout, fin * fout, fout * t, fin * t):
            quant = up(quant + n // 2)
            quant = up(quant + n // 32)
        got = lib.mx_linear_backward_workspace_bytes(t, fin, fout)
        assert got >= quant and got % 256 == 0
        assert (got - quant) % (4 * fin) == 0        # partials are whole [rows, in] fp32 slabs
    assert lib.mx_linear_backward_workspace_bytes(-1, 1, 1) == 0


def test_linear_backward_ex_validation():
    """mx_linear_backward_ex: flags, mode, g, shapes, NULL and alignment are all
    checked before any HIP call."""
    lib = _lib()
    f = lib.mx_linear_backward_ex
    rs, bf, acc = binding.MX_MODE_RHT_SR, binding.MX_BWD_DX_BF16, binding.MX_BWD_ACCUMULATE
    args = (FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 64, 0)
    assert f(*args, rs, 4, None) == -9                      # unknown flag bit
    assert f(*args, rs, 0x80000000, None) == -9
    assert f(*args, 9, 0, None) == -8                       # unknown mode
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 64, 40, 0, rs, 0, None) == -2
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 96, 64, 64, 64, 0, rs, 0, None) == -3     # g | T
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, 64, 96, 64, 0, rs, 0, None) == -3     # g | out
    assert f(FAKE, FAKE, FAKE, None, FAKE, FAKE, 64, 64, 64, 64, 0, rs, 0, None) == -1     # dX
    assert f(FAKE, FAKE, FAKE, FAKE, None, FAKE, 64, 64, 64, 64, 0, rs, acc, None) == -1   # dW
    assert f(None, FAKE, FAKE, FAKE, FAKE, None, 64, 64, 64, 64, 0, rs, 0, None) == -1     # dY
    # dX alignment: 4 bytes for float32, 2 for bf16; db 4 bytes
    assert f(FAKE, FAKE, FAKE, FAKE + 2, FAKE, FAKE, 64, 64, 64, 64, 0, rs, 0, None) == -4
    assert f(FAKE, FAKE, FAKE, FAKE + 1, FAKE, FAKE, 64, 64, 64, 64, 0, rs, bf, None) == -4
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, 64, 64, 64, 64, 0, rs, 0, None) == -4
    # nothing to compute: no outputs exist (in == 0) and no bias
    assert f(FAKE, None, None, None, None, None, 64, 0, 64, 64, 0, rs, bf | acc, None) == 0
    assert f(None, None, None, None, None, None, 64, 0, 0, 64, 0, rs, 0, None) == 0
    # db alone (in == 0) still needs dY
    assert f(None, None, None, None, None, FAKE, 64, 0, 64, 64, 0, rs, 0, None) == -1


def test_linear_backward_ex_workspace_bytes():
    """With db the workspace adds the block sums: (T / block) * out float32 values,
    block = g with the RHT and 32 without; without db it is mx_linear_backward's."""
    lib = _lib()
    w0 = lib.mx_linear_backward_workspace_bytes
    wx = lib.mx_linear_backward_ex_workspace_bytes
    def up(v):
        return (v + 255) // 256 * 256
    for t, fin, fout, g in ((4096, 1024, 3072, 64), (256, 256, 256, 128), (64, 40, 64, 32)):
        base = w0(t, fin, fout)
        assert wx(t, fin, fout, g, binding.MX_MODE_RHT_SR, 0) == base
        assert wx(t, fin, fout, g, binding.MX_MODE_RHT_SR, 1) == base + up(t // g * fout * 4)
        assert wx(t, fin, fout, 0, binding.MX_MODE_SR, 1) == base + up(t // 32 * fout * 4)
    assert wx(64, 64, 64, 48, binding.MX_MODE_RHT_SR, 1) == 0
    assert wx(64, 64, 64, 64, 7, 1) == 0


# --- Python binding argument checks (no GPU: CPU tensors never reach the library) ---

def _t(shape, dtype):
    import torch
    return torch.zeros(shape, dtype=dtype)


def test_binding_rejects_mismatched_shapes_and_dtypes():
    import torch
    u8, f32, b16 = torch.uint8, torch.float32, torch.bfloat16
    m, n, k = 8, 16, 64
    ok = dict(a_codes=_t((m, k // 2), u8), a_scales=_t((m, k // 32), u8), b_codes=_t((n, k // 2), u8),
              b_scales=_t((n, k // 32), u8), c=_t((m, n), f32))
    bad = [("b_codes", _t((n, k // 2 + 1), u8)), ("a_scales", _t((m, k // 32 + 1), u8)),
           ("b_scales", _t((n + 1, k // 32), u8)), ("c", _t((m, n - 1), f32)), ("c", _t((m, n), b16)),
           ("a_codes", _t((m, k // 2), torch.int8))]
    for name, t in bad:
        args = dict(ok, **{name: t})
        with pytest.raises(ValueError, match=name.split("_")[0]):
            binding.mx_gemm_f4(**args)
    t_, fin, fout = 64, 32, 64
    dy, x, w = _t((t_, fout), b16), _t((t_, fin), b16), _t((fout, fin), b16)
    dx, dw, db = _t((t_, fin), f32), _t((fout, fin), f32), _t((fout,), f32)
    for args in ((dy, _t((t_ + 1, fin), b16), w, dx, dw), (dy, x, _t((fout, fin + 1), b16), dx, dw),
                 (dy, x, w, _t((t_, fin + 1), f32), dw), (dy, x, w, dx, _t((fout, fin), torch.float64)),
                 (dy, x, w, _t((t_, fin), b16), dw)):
        with pytest.raises(ValueError):
            binding.mx_linear_backward(*args, 64, 0)
    with pytest.raises(ValueError, match="db"):
        binding.mx_linear_backward_ex(dy, x, w, dx, dw, _t((fout + 1,), f32), 64, 0)
    # bf16 dX with MX_BWD_DX_BF16: a float32 dX of the right shape is the wrong kind
    with pytest.raises(ValueError, match="dx"):
        binding.mx_linear_backward_ex(dy, x, w, dx, dw, db, 64, 0, binding.MX_MODE_RHT_SR, binding.MX_BWD_DX_BF16)
    with pytest.raises(ValueError, match="codes"):
        binding.mx_rht_sr_quantize(dy, _t((t_, fout // 2 - 1), u8), _t((t_, fout // 32), u8), 64, 0)
    with pytest.raises(ValueError, match="scales"):
        # stored [cols = 32, rows = 64]: logical [64, 32], so codes [64, 16] and scales [64, 1]
        binding.mx_rht_sr_quantize_t(_t((32, 64), b16), _t((64, 16), u8), _t((64, 2), u8), 32, 0)
    with pytest.raises(ValueError, match="contiguous"):
        binding.mx_rht_sr_quantize(_t((fout, t_), b16).t(), _t((t_, fout // 2), u8), _t((t_, fout // 32), u8),
                                   64, 0)


def test_binding_rejects_host_tensors():
    """Well-formed arguments that live in host memory are refused before the library is called."""
    import torch
    dy = _t((64, 64), torch.bfloat16)
    with pytest.raises(ValueError, match="current GPU"):
        binding.mx_rht_sr_quantize(dy, _t((64, 32), torch.uint8), _t((64, 2), torch.uint8), 64, 0)


def test_capture_status_is_declared():
    text = open(HEADER).read()
    assert re.search(r"MX_ERR_CAPTURE\s*=\s*-10", text)
    assert binding._STATUS[-10] == "MX_ERR_CAPTURE"


def test_binding_loads_one_hip_runtime():
    """load_library() in a fresh process, before anything imports torch: the
    library must bind to the HIP runtime torch loads, so the process maps one
    libamdhip64 (two runtimes do not share devices or streams)."""
    import subprocess
    import sys
    _lib()
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import paper_2502_20586_amd.binding as b\n"
            "b.load_library()\n"
            "print(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    runtimes = eval(out.stdout.strip().splitlines()[-1])
    assert len(runtimes) == 1, runtimes
