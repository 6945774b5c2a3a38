"""mx_linear_backward_noalloc captured into a HIP graph (torch.cuda.graph) and
replayed: the entry point for callers that cannot allocate, which is what code
under graph capture needs. Each replay runs on new inputs copied into the
captured buffers, with eager work (copies and a plain mx_linear_backward) and
synchronisations between replays, and must equal mx_linear_backward on the
same inputs bit for bit. Two shapes: one whose dW GEMM is split along K (the
reduction kernel is captured too) and one that is not.
"""

import numpy as np
import pytest

from gpu_util import host, note, to_dev, torch_gpu
from workloads import matrix

pytestmark = pytest.mark.gpu


def _inputs(t, fin, fout, seed):
    dy = matrix((t, fout), [seed, 0], dist="t3", scale=1e-3, outlier_p=0.01, outlier_factor=100.0)
    x = matrix((t, fin), [seed, 1])
    w = matrix((fout, fin), [seed, 2], scale=0.02)
    return dy, x, w


@pytest.mark.parametrize("t,fin,fout,g", [(1024, 384, 768, 64), (4096, 128, 128, 64)])
def test_noalloc_graph_replays_equal_eager_calls(t, fin, fout, g):
    torch = torch_gpu()
    import paper_2502_20586_amd as mx
    seed = 0x6A0F_0000_0000_0000 | t
    dy, x, w = _inputs(t, fin, fout, 500)
    d_dy, d_x, d_w = to_dev(dy), to_dev(x), to_dev(w)
    dx = torch.full((t, fin), float("nan"), dtype=torch.float32, device="cuda")
    dw = torch.full((fout, fin), float("nan"), dtype=torch.float32, device="cuda")
    note(f"graph noalloc T={t} in={fin} out={fout} g={g}: eager call")
    mx.mx_linear_backward_noalloc(d_dy, d_x, d_w, dx, dw, g, seed)   # looks up the scratch address
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    note("graph noalloc: capture")
    with torch.cuda.graph(graph, stream=side):
        mx.mx_linear_backward_noalloc(d_dy, d_x, d_w, dx, dw, g, seed)
    torch.cuda.synchronize()
    ref_dx = torch.empty_like(dx)
    ref_dw = torch.empty_like(dw)
    for k in range(3):
        dy, x, w = _inputs(t, fin, fout, 600 + k)
        d_dy.copy_(to_dev(dy))
        d_x.copy_(to_dev(x))
        d_w.copy_(to_dev(w))
        dx.fill_(float("nan"))
        dw.fill_(float("nan"))
        torch.cuda.synchronize()
        note(f"graph noalloc: replay {k}")
        graph.replay()
        torch.cuda.synchronize()
        got_dx, got_dw = host(dx), host(dw)
        mx.mx_linear_backward(d_dy, d_x, d_w, ref_dx, ref_dw, g, seed)
        torch.cuda.synchronize()
        assert np.all(np.isfinite(got_dx)) and np.all(np.isfinite(got_dw))
        assert np.array_equal(got_dx, host(ref_dx)) and np.array_equal(got_dw, host(ref_dw))
