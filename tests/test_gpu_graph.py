"""The CCL path under HIP graph capture: pack -> GEMM -> GEMM -> unpack of a
small FFN step, captured once and replayed several times with eager work and
synchronisation in between. Every replay must equal the eager run bit for
bit (the kernels allocate nothing and use no memset, so they can be
captured)."""
import numpy as np
import pytest

import workloads as W
from paper_2606_11718_amd import ccl
from tests.helpers import from_dev, to_dev

pytestmark = pytest.mark.gpu


def test_ffn_step_graph_replays_match_eager():
    import torch

    T, D, F, G, Gr, P = 1024, 512, 1536, 8, 2, 4096
    up = ccl.ccl_plan(T, F, D, G, Gr, P)
    down = ccl.ccl_plan(T, D, F, G, Gr, P)
    size = lambda p, op: ccl.ccl_plan_layout(p, op).total_bytes // 2  # noqa: E731
    X = to_dev(W.draw_array(301, T, D, "normal", 1.0))
    W1 = to_dev(W.draw_array(302, D, F, "normal", 0.03))
    W2 = to_dev(W.draw_array(303, F, D, "normal", 0.02))
    dev = X.device
    Xc, W1c, Hc = (torch.empty(size(up, op), dtype=torch.int16, device=dev)
                   for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    W2c, Yc = (torch.empty(size(down, op), dtype=torch.int16, device=dev) for op in (ccl.CCL_B, ccl.CCL_C))
    Y = torch.empty(T, D, dtype=torch.int16, device=dev)
    ccl.ccl_pack(up, ccl.CCL_B, W1, F, 0, W1c)
    ccl.ccl_pack(down, ccl.CCL_B, W2, D, 0, W2c)

    def step():
        ccl.ccl_pack(up, ccl.CCL_A, X, D, 0, Xc)
        ccl.ccl_gemm(up, Xc, W1c, Hc)
        ccl.ccl_gemm_scaled(down, 0.5, Hc, W2c, 0.0, Yc)
        ccl.ccl_unpack(down, ccl.CCL_C, Yc, Y, D)

    step()
    eager = from_dev(Y).copy()
    print("graph capture of the FFN step", flush=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step()                                   # warm-up on the capture stream
        torch.cuda.synchronize()
        Y.fill_(0)
        with torch.cuda.graph(graph, stream=side):
            step()
    torch.cuda.synchronize()
    for rep in range(3):
        Y.fill_(0)
        Hc.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(Y), eager), f"replay {rep}"
