"""ctypes binding of libmxfp4.so.

Names and argument order follow the C ABI (include/mxfp4.h). Tensors are torch
tensors on the current HIP device; torch supplies device memory and the current
stream, nothing else. bf16 inputs may be passed as torch.bfloat16 or as
torch.int16/uint16 bit patterns.
"""

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
_LIB = None

_STATUS = {
    0: "MX_OK", -1: "MX_ERR_NULL", -2: "MX_ERR_G", -3: "MX_ERR_SHAPE", -4: "MX_ERR_ALIGN",
    -5: "MX_ERR_HIP", -6: "MX_ERR_NOMEM", -7: "MX_ERR_DEVICE", -8: "MX_ERR_MODE", -9: "MX_ERR_FLAGS",
    -10: "MX_ERR_CAPTURE", -11: "MX_ERR_TOO_LARGE",
}

# Scratch held by mx_linear_backward_noalloc on each GPU (include/mxfp4.h).
MX_NOALLOC_SCRATCH_BYTES = 64 << 20

# Quantiser modes (include/mxfp4.h, enum mx_mode): the method and the ablation
# rows of Table 2.
MX_MODE_RHT_SR, MX_MODE_SR, MX_MODE_RHT_NR, MX_MODE_NR = 0, 1, 2, 3
# The cheaper-noise variant (8-bit dither; a deliberate change of the rounding rule).
MX_MODE_RHT_SR8 = 4

# Options of mx_linear_backward_ex (include/mxfp4.h, enum mx_backward_flags).
MX_BWD_DX_BF16, MX_BWD_ACCUMULATE = 1, 2


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("work", ctypes.c_double), ("work_is_flops", ctypes.c_int)]


class MxError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(msg)
        self.status = status


def lib_path():
    return os.path.join(PKG, "libmxfp4.so")


def load_library():
    """Load libmxfp4.so from the package directory (built by build.py). Raises if absent.

    torch is imported first: the library then binds to the HIP runtime that
    torch has loaded (it needs libamdhip64.so.7, which torch's copy provides
    under that name). Loaded the other way round, the library would pull in
    the system's HIP runtime and torch its own, and two runtimes in one
    process do not share devices or streams (the library's calls then fail
    with MX_ERR_HIP)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    import torch  # noqa: F401  (see above)
    path = lib_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2502_20586_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i64, u64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int
    lib.mx_status_string.restype = ctypes.c_char_p
    lib.mx_status_string.argtypes = [ci]
    lib.mx_rht_sr_quantize.restype = ci
    lib.mx_rht_sr_quantize.argtypes = [vp, vp, vp, i64, i64, ci, u64, vp]
    lib.mx_rht_sr_quantize_t.restype = ci
    lib.mx_rht_sr_quantize_t.argtypes = [vp, vp, vp, i64, i64, ci, u64, vp]
    lib.mx_quantize.restype = ci
    lib.mx_quantize.argtypes = [vp, vp, vp, i64, i64, ci, u64, ci, ci, vp]
    lib.mx_linear_backward_mode.restype = ci
    lib.mx_linear_backward_mode.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ci, u64, ci, vp]
    lib.mx_quantize_pair.restype = ci
    lib.mx_quantize_pair.argtypes = [vp, vp, vp, vp, vp, i64, i64, ci, u64, u64, ci, vp]
    lib.mx_gemm_f4_workspace_bytes.restype = i64
    lib.mx_gemm_f4_workspace_bytes.argtypes = [i64, i64, i64]
    lib.mx_release_workspace.restype = ci
    lib.mx_release_workspace.argtypes = [vp]
    lib.mx_gemm_f4.restype = ci
    lib.mx_gemm_f4.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, vp]
    lib.mx_linear_backward.restype = ci
    lib.mx_linear_backward.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ci, u64, vp]
    lib.mx_linear_backward_noalloc.restype = ci
    lib.mx_linear_backward_noalloc.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, ci, u64, vp]
    lib.mx_linear_backward_workspace_bytes.restype = i64
    lib.mx_linear_backward_workspace_bytes.argtypes = [i64, i64, i64]
    lib.mx_linear_backward_ex.restype = ci
    lib.mx_linear_backward_ex.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, ci, u64, ci, ctypes.c_uint, vp]
    lib.mx_linear_backward_ex_workspace_bytes.restype = i64
    lib.mx_linear_backward_ex_workspace_bytes.argtypes = [i64, i64, i64, ci, ci, ci]
    lib.mx_profile_start.restype = ci
    lib.mx_profile_start.argtypes = []
    lib.mx_profile_stop.restype = ci
    lib.mx_profile_stop.argtypes = [ctypes.POINTER(KernelStat), ci, ctypes.POINTER(ci)]
    lib.mx_measure_mfma_peak.restype = ci
    lib.mx_measure_mfma_peak.argtypes = [ci, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    _LIB = lib
    return lib


def _check(status):
    if status != 0:
        lib = load_library()
        raise MxError(status, lib.mx_status_string(status).decode())


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# Argument checks. The library trusts the sizes it is given: an output tensor
# smaller than the sizes say would be written past its end on the device. So
# every wrapper checks each tensor's dtype, shape and layout against the sizes
# it passes, and that all tensors live on the current GPU, before calling the
# library; a mismatch raises ValueError and nothing is called.

def _dtypes(kind):
    import torch
    return {
        "bf16": (torch.bfloat16, torch.int16, torch.uint16),     # bf16 values or their bit patterns
        "u8": (torch.uint8,),
        "f32": (torch.float32,),
    }[kind]


def _arg(t, name, kind, shape):
    """Checks one tensor argument; returns its device pointer (None for an empty tensor)."""
    if t is None:
        raise ValueError(f"{name}: a tensor is required")
    if t.dtype not in _dtypes(kind):
        raise ValueError(f"{name}: dtype {t.dtype} is not one of {_dtypes(kind)}")
    if tuple(t.shape) != tuple(int(d) for d in shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: tensors must be contiguous (row-major)")
    return t


def _ptrs(*tensors):
    """Device pointers of checked tensors, after checking they are all on the current GPU."""
    import torch
    live = [t for t in tensors if t is not None]
    for t in live:
        if t.device.type != "cuda":
            raise ValueError(f"tensor on {t.device}: the library takes tensors on the current GPU")
    if live:
        cur = torch.cuda.current_device()
        for t in live:
            if t.device.index != cur:
                raise ValueError(f"tensor on {t.device}, but the current device is cuda:{cur}")
    return [None if t is None else (t.data_ptr() or None) for t in tensors]


def _two_d(t, name):
    if t is None or t.dim() != 2:
        raise ValueError(f"{name}: a 2-D tensor is required")
    return t.shape


def quantized_shapes(rows, cols):
    """(codes shape, scales shape) of an MXFP4 matrix with logical shape [rows, cols]."""
    return (rows, cols // 2), (rows, cols // 32)


def _quant_args(x, codes, scales, transposed):
    if transposed:
        cols, rows = _two_d(x, "x_t")
    else:
        rows, cols = _two_d(x, "x")
    cs, ss = quantized_shapes(rows, cols)
    _arg(x, "x_t" if transposed else "x", "bf16", x.shape)
    _arg(codes, "codes", "u8", cs)
    _arg(scales, "scales", "u8", ss)
    return rows, cols, _ptrs(x, codes, scales)


def mx_rht_sr_quantize(x, codes, scales, g, seed, stream=None):
    """Quantise row-major bf16 x [rows, cols] (blocks along cols) into codes/scales (uint8)."""
    rows, cols, p = _quant_args(x, codes, scales, False)
    _check(load_library().mx_rht_sr_quantize(*p, rows, cols, g, seed & 0xFFFFFFFFFFFFFFFF, _stream(stream)))


def mx_rht_sr_quantize_t(x_t, codes, scales, g, seed, stream=None):
    """Quantise the transpose of bf16 x_t [cols, rows]: logical matrix [rows, cols]."""
    rows, cols, p = _quant_args(x_t, codes, scales, True)
    _check(load_library().mx_rht_sr_quantize_t(*p, rows, cols, g, seed & 0xFFFFFFFFFFFFFFFF, _stream(stream)))


def mx_quantize(x, codes, scales, g, seed, mode, transposed=False, stream=None):
    """Quantise in any mode (MX_MODE_*). transposed=False: x is the row-major [rows, cols]
    matrix; transposed=True: x is stored [cols, rows] and the logical matrix is its transpose."""
    rows, cols, p = _quant_args(x, codes, scales, bool(transposed))
    _check(load_library().mx_quantize(*p, rows, cols, g, seed & 0xFFFFFFFFFFFFFFFF, mode, 1 if transposed else 0,
                                      _stream(stream)))


def mx_quantize_pair(x, codes, scales, codes_t, scales_t, g, seed, seed_t, mode=0, stream=None):
    """Both quantisations of row-major bf16 x [rows, cols] in one pass: codes/scales of x
    (blocks along cols, seed) and codes_t/scales_t of x^T [cols, rows] (blocks along rows,
    seed_t)."""
    rows, cols = _two_d(x, "x")
    _arg(x, "x", "bf16", (rows, cols))
    cs, ss = quantized_shapes(rows, cols)
    cst, sst = quantized_shapes(cols, rows)
    _arg(codes, "codes", "u8", cs)
    _arg(scales, "scales", "u8", ss)
    _arg(codes_t, "codes_t", "u8", cst)
    _arg(scales_t, "scales_t", "u8", sst)
    _check(load_library().mx_quantize_pair(*_ptrs(x, codes, scales, codes_t, scales_t), rows, cols, g,
                                           seed & 0xFFFFFFFFFFFFFFFF, seed_t & 0xFFFFFFFFFFFFFFFF, mode,
                                           _stream(stream)))


def mx_gemm_f4(a_codes, a_scales, b_codes, b_scales, c, stream=None):
    """C[M, N] (float32) = deq(A) @ deq(B)^T for MXFP4 operands A [M, K], B [N, K]."""
    m, kh = _two_d(a_codes, "a_codes")
    n = _two_d(b_codes, "b_codes")[0]
    k = 2 * kh
    _arg(a_codes, "a_codes", "u8", (m, kh))
    _arg(a_scales, "a_scales", "u8", (m, k // 32))
    _arg(b_codes, "b_codes", "u8", (n, kh))
    _arg(b_scales, "b_scales", "u8", (n, k // 32))
    _arg(c, "c", "f32", (m, n))
    _check(load_library().mx_gemm_f4(*_ptrs(a_codes, a_scales, b_codes, b_scales, c), m, n, k, _stream(stream)))


def mx_gemm_f4_workspace_bytes(m, n, k):
    """Bytes of workspace mx_gemm_f4 needs for an [m, k] x [n, k] product."""
    return int(load_library().mx_gemm_f4_workspace_bytes(m, n, k))


def mx_release_workspace(stream=None):
    """Free the library's workspace for the current device and stream, in stream order."""
    _check(load_library().mx_release_workspace(_stream(stream)))


def _backward_args(dy, x, w, dx, dw, db=None, dx_kind="f32"):
    t, out_f = _two_d(dy, "dy")
    in_f = _two_d(x, "x")[1]
    _arg(dy, "dy", "bf16", (t, out_f))
    _arg(x, "x", "bf16", (t, in_f))
    _arg(w, "w", "bf16", (out_f, in_f))
    _arg(dx, "dx", dx_kind, (t, in_f))
    _arg(dw, "dw", "f32", (out_f, in_f))
    if db is not None:
        _arg(db, "db", "f32", (out_f,))
    return t, in_f, out_f


def mx_linear_backward(dy, x, w, dx, dw, g, seed, stream=None):
    """Algorithm 3: dX = 16/(9g) Q(dY) Q(W^T)^T, dW = 16/(9g) Q(dY^T) Q(x^T)^T (float32 outputs)."""
    t, in_f, out_f = _backward_args(dy, x, w, dx, dw)
    _check(load_library().mx_linear_backward(*_ptrs(dy, x, w, dx, dw), t, in_f, out_f, g,
                                             seed & 0xFFFFFFFFFFFFFFFF, _stream(stream)))


def mx_linear_backward_noalloc(dy, x, w, dx, dw, g, seed, stream=None):
    """mx_linear_backward with its scratch in the library's fixed per-GPU array (no allocation;
    problems needing more than MX_NOALLOC_SCRATCH_BYTES raise MX_ERR_TOO_LARGE)."""
    t, in_f, out_f = _backward_args(dy, x, w, dx, dw)
    _check(load_library().mx_linear_backward_noalloc(*_ptrs(dy, x, w, dx, dw), t, in_f, out_f, g,
                                                     seed & 0xFFFFFFFFFFFFFFFF, _stream(stream)))


def mx_linear_backward_mode(dy, x, w, dx, dw, g, seed, mode, stream=None):
    """mx_linear_backward with the operands quantised in mode `mode` (MX_MODE_*)."""
    t, in_f, out_f = _backward_args(dy, x, w, dx, dw)
    _check(load_library().mx_linear_backward_mode(*_ptrs(dy, x, w, dx, dw), t, in_f, out_f, g,
                                                  seed & 0xFFFFFFFFFFFFFFFF, mode, _stream(stream)))


def mx_linear_backward_workspace_bytes(t, in_features, out_features):
    return int(load_library().mx_linear_backward_workspace_bytes(t, in_features, out_features))


def mx_linear_backward_ex(dy, x, w, dx, dw, db, g, seed, mode=MX_MODE_RHT_SR, flags=0, stream=None):
    """Backward of y = x W^T + b: dX and dW by Algorithm 3 (dx float32, or bf16 with
    MX_BWD_DX_BF16), db = column sums of dY (db=None: no bias); MX_BWD_ACCUMULATE adds
    dW and db to the tensors' contents."""
    t, in_f, out_f = _backward_args(dy, x, w, dx, dw, db, "bf16" if flags & MX_BWD_DX_BF16 else "f32")
    _check(load_library().mx_linear_backward_ex(*_ptrs(dy, x, w, dx, dw, db), t, in_f, out_f, g,
                                                seed & 0xFFFFFFFFFFFFFFFF, mode, flags, _stream(stream)))


def mx_linear_backward_ex_workspace_bytes(t, in_features, out_features, g, mode=MX_MODE_RHT_SR, with_db=True):
    return int(load_library().mx_linear_backward_ex_workspace_bytes(t, in_features, out_features, g, mode,
                                                                    1 if with_db else 0))


def mx_profile_start():
    """Start tracing the library's kernel launches (HIP events on their streams)."""
    _check(load_library().mx_profile_start())


def mx_profile_stop():
    """Stop tracing; returns {kernel: dict(launches, total_ms, work, work_is_flops)}."""
    lib = load_library()
    cap = 64
    arr = (KernelStat * cap)()
    n = ctypes.c_int(0)
    _check(lib.mx_profile_stop(arr, cap, ctypes.byref(n)))
    out = {}
    for i in range(min(n.value, cap)):
        s = arr[i]
        out[s.name.decode()] = {"launches": int(s.launches), "total_ms": float(s.total_ms),
                                "work": float(s.work), "work_is_flops": bool(s.work_is_flops)}
    return out


def mx_measure_mfma_peak(rounds=2000):
    """(TFLOP/s, clock GHz) of FP4 MFMAs issued back to back from registers on every CU:
    the rate the GEMM can reach at best. Synchronises; takes about half a second."""
    tf, ghz = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(load_library().mx_measure_mfma_peak(rounds, ctypes.byref(tf), ctypes.byref(ghz)))
    return tf.value, ghz.value
