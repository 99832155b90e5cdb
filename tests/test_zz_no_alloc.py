"""ccl_gemm_splitk_noalloc: the split-K GEMM with its fp32 partials in the
library's static device scratch instead of a caller workspace.

Two calls in a row on one GPU, the second with a smaller input (so the
scratch still holds the first call's larger partials): each must give the
same C as ccl_gemm_splitk with a caller workspace (same kernels, ranges and
summation order, so bit for bit) and meet the GEMM bar against the fp64
oracle (relative Frobenius <= 5e-3, max abs <= 1e-2 max|ref| for bf16 C;
relative Frobenius <= 1e-4 for fp32 C).
"""
import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import torch_mod

pytestmark = pytest.mark.gpu


def _to_dev(a: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1)).to("cuda")


def _dev_bytes(n: int, value: int):
    torch = torch_mod()
    return torch.full((max(n, 1),), value, dtype=torch.uint8, device="cuda")


def _both(M, N, K, G, Gr, a_trans, splits, c_type, alpha, beta, seed):
    A = W.draw_array(seed, *((K, M) if a_trans else (M, K)), "normal", 1.0)
    B = W.draw_array(seed + 1, K, N, "normal", 0.02)
    plan = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ccl.CCL_DT_BF16, c_type)
    gr, gc = ccl.ccl_plan_grid(plan)
    ranges, need = ccl.ccl_gemm_splitk_workspace(plan, splits)
    print(f"noalloc splitk {M}x{N}x{K} grid {gr}x{gc} splits={splits} -> {ranges} ws={need} "
          f"c={c_type} alpha={alpha} beta={beta}", flush=True)
    assert ranges > 1 and 0 < need <= ccl.CCL_SCRATCH_BYTES
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc = _dev_bytes(la.total_bytes, 0), _dev_bytes(lb.total_bytes, 0)
    ccl.ccl_pack(plan, ccl.CCL_A, _to_dev(A), A.shape[1], a_trans, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, _to_dev(B), N, 0, Bc)
    cdt = np.uint32 if c_type == ccl.CCL_DT_FP32 else np.uint16
    C0 = W.draw_array(seed + 2, M, N, "normal", 1.0)
    C0 = (OG.decode_bf16(C0).astype(np.float32).view(np.uint32) if cdt == np.uint32 else C0)
    C0_ccl = OL.pack(C0, gr, gc, 4096)
    C_ws, C_static = _to_dev(C0_ccl), _to_dev(C0_ccl)
    ws = _dev_bytes(need, 0xFF)
    ccl.ccl_gemm_splitk(plan, alpha, Ac, Bc, beta, C_ws, splits, ws, need)
    ccl.ccl_gemm_splitk_noalloc(plan, alpha, Ac, Bc, beta, C_static, splits)
    torch_mod().cuda.synchronize()
    got_ws = C_ws.cpu().numpy().view(cdt)
    got_static = C_static.cpu().numpy().view(cdt)
    assert np.array_equal(got_static, got_ws)
    bits = OL.unpack(got_static, M, N, gr, gc, 4096)
    C = bits.view(np.float32).astype(np.float64) if cdt == np.uint32 else OG.decode_bf16(bits)
    A_l = np.ascontiguousarray(A.T) if a_trans else A
    C0_val = C0.view(np.float32) if cdt == np.uint32 else C0
    err = OG.errors(C, OG.gemm_scaled_fp64(A_l, B, C0_val, alpha, beta))
    print("errors", err, flush=True)
    if cdt == np.uint32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_noalloc_splitk_equals_workspace_splitk_on_two_calls(c_type):
    # Qwen3 dW_down (A = H^T stored transposed), 4 K ranges: 25 MB of partials
    _both(768, 2048, 4096, 8, 1, 1, 4, c_type, 1.0, 0.0, 7100)
    # then a smaller GEMM with C read (alpha A B + beta C): 2.6 MB of partials
    _both(256, 512, 1280, 4, 2, 0, 5, c_type, 0.5, -1.0, 7200)
