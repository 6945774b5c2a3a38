"""Graph capture is refused by every entry point that enqueues work.

The entry points may allocate or free their workspace in stream order, which a
HIP graph cannot replay, and a graph would keep a workspace address that a
later call may free. On a stream that is being captured they return
MX_ERR_CAPTURE (-10) and enqueue nothing. The test begins a capture on a fresh
stream, calls each entry point on it, ends the capture and destroys the empty
graph without instantiating or replaying it; then the same stream runs a
backward pass normally.
"""

import ctypes

import pytest

from gpu_util import note, torch_gpu, to_dev
from workloads import matrix

pytestmark = pytest.mark.gpu

MX_ERR_CAPTURE = -10
CAPTURE_MODE_THREAD_LOCAL = 1    # hipStreamCaptureModeThreadLocal


def _hip_runtime():
    """The HIP runtime library this process has loaded (the one torch and the library use)."""
    paths = sorted({l.split()[-1] for l in open("/proc/self/maps").read().splitlines() if "libamdhip64" in l})
    assert paths, "no HIP runtime loaded"
    hip = ctypes.CDLL(paths[0])
    hip.hipStreamBeginCapture.argtypes = [ctypes.c_void_p, ctypes.c_int]
    hip.hipStreamEndCapture.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    hip.hipGraphDestroy.argtypes = [ctypes.c_void_p]
    return hip


def test_entry_points_refuse_a_capturing_stream():
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    t, fin, fout, g, seed = 256, 128, 256, 64, 0xCA97_0000_0000_0001
    dy, x, w = matrix((t, fout), 1), matrix((t, fin), 2), matrix((fout, fin), 3, scale=0.02)
    ddy, dx_in, dw_in = to_dev(dy), to_dev(x), to_dev(w)
    dx = torch.full((t, fin), 7.0, device="cuda")
    dw = torch.full((fout, fin), 7.0, device="cuda")
    db = torch.full((fout,), 7.0, device="cuda")
    codes = torch.zeros((t, fout // 2), dtype=torch.uint8, device="cuda")
    scales = torch.zeros((t, fout // 32), dtype=torch.uint8, device="cuda")
    codes_t = torch.zeros((fout, t // 2), dtype=torch.uint8, device="cuda")
    scales_t = torch.zeros((fout, t // 32), dtype=torch.uint8, device="cuda")
    c = torch.full((t, fout), 7.0, device="cuda")
    torch.cuda.synchronize()

    calls = {
        "mx_rht_sr_quantize": lambda s: mx.mx_rht_sr_quantize(ddy, codes, scales, g, seed, stream=s),
        "mx_rht_sr_quantize_t": lambda s: mx.mx_rht_sr_quantize_t(ddy, codes_t, scales_t, g, seed, stream=s),
        "mx_quantize": lambda s: mx.mx_quantize(ddy, codes, scales, g, seed, mx.MX_MODE_NR, stream=s),
        "mx_quantize_pair": lambda s: mx.mx_quantize_pair(ddy, codes, scales, codes_t, scales_t, g, seed,
                                                          seed ^ 2, stream=s),
        "mx_gemm_f4": lambda s: mx.mx_gemm_f4(codes, scales, codes, scales, c, stream=s),
        "mx_release_workspace": lambda s: mx.mx_release_workspace(stream=s),
        "mx_linear_backward": lambda s: mx.mx_linear_backward(ddy, dx_in, dw_in, dx, dw, g, seed, stream=s),
        "mx_linear_backward_mode": lambda s: mx.mx_linear_backward_mode(ddy, dx_in, dw_in, dx, dw, g, seed,
                                                                        mx.MX_MODE_SR, stream=s),
        "mx_linear_backward_ex": lambda s: mx.mx_linear_backward_ex(ddy, dx_in, dw_in, dx, dw, db, g, seed,
                                                                    mx.MX_MODE_RHT_SR, mx.MX_BWD_ACCUMULATE,
                                                                    stream=s),
    }
    hip = _hip_runtime()
    s = torch.cuda.Stream()
    handle = ctypes.c_void_p(s.cuda_stream)
    note("capture: begin on a fresh stream")
    assert hip.hipStreamBeginCapture(handle, CAPTURE_MODE_THREAD_LOCAL) == 0
    statuses = {}
    try:
        for name, fn in calls.items():
            note(f"capture: {name}")
            try:
                fn(s)
                statuses[name] = 0
            except mx.MxError as e:
                statuses[name] = e.status
    finally:
        graph = ctypes.c_void_p()
        rc = hip.hipStreamEndCapture(handle, ctypes.byref(graph))
        if graph.value:
            hip.hipGraphDestroy(graph)
    assert rc == 0
    assert statuses == {name: MX_ERR_CAPTURE for name in calls}, statuses
    torch.cuda.synchronize()
    # Nothing was enqueued: the outputs still hold what they held.
    for tns in (dx, dw, db, c):
        assert torch.all(tns == 7.0)
    assert torch.all(codes == 0) and torch.all(scales == 0)
    assert torch.all(codes_t == 0) and torch.all(scales_t == 0)

    note("capture: the stream works normally afterwards")
    mx.mx_linear_backward(ddy, dx_in, dw_in, dx, dw, g, seed, stream=s)
    ref_dx = torch.empty_like(dx)
    ref_dw = torch.empty_like(dw)
    s.synchronize()
    mx.mx_linear_backward(ddy, dx_in, dw_in, ref_dx, ref_dw, g, seed)
    torch.cuda.synchronize()
    assert torch.equal(dx, ref_dx) and torch.equal(dw, ref_dw)
    assert not torch.all(dx == 7.0)
