"""GPU parity of ccl_pack / ccl_unpack with the oracle's CCL map: bit-exact.

Every workload operand is packed from its stored form (row-major or stored
transpose) and compared with the oracle's pack of the logical operand;
padding must keep its canary, and unpack must return the source bits.
"""
import numpy as np
import pytest

import workloads as W
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import CANARY, dev_full, from_dev, to_dev, with_ld

pytestmark = pytest.mark.gpu

OPS = {"A": ccl.CCL_A, "B": ccl.CCL_B, "C": ccl.CCL_C}


def _check_pack(stored: np.ndarray, trans: int, op: str, M, N, K, G, Gr, P, ld=None):
    """stored: the tensor as it sits in memory (the transpose if trans)."""
    plan = ccl.ccl_plan(M, N, K, G, Gr, P)
    gr, gc = ccl.ccl_plan_grid(plan)
    lay = ccl.ccl_plan_layout(plan, OPS[op])
    logical = stored.T if trans else stored
    R, Cc = logical.shape
    assert (R, Cc) == OL.operand_shape(op, M, N, K)
    ld = ld or stored.shape[1]
    src = to_dev(with_ld(stored, ld) if ld != stored.shape[1] else stored)
    dst = dev_full(lay.total_bytes // 2)
    print(f"pack {op} {R}x{Cc} grid {gr}x{gc} P={P} trans={trans} ld={ld}", flush=True)
    ccl.ccl_pack(plan, OPS[op], src, ld, trans, dst)
    got = from_dev(dst)
    ref = OL.pack_reshape(np.ascontiguousarray(logical), gr, gc, P)
    if lay.total_bytes != lay.strip_bytes * gr * gc:
        pad = OL.padding_mask(R, Cc, gr, gc, P)
        assert np.array_equal(got[~pad], ref[~pad])
        assert np.all(got[pad] == CANARY)
    else:
        assert np.array_equal(got, ref)
    return plan, dst, logical


def _check_unpack(plan, op, dst, logical, ld=None):
    R, Cc = logical.shape
    ld = ld or Cc
    out = dev_full(R * ld, 0x1234)
    ccl.ccl_unpack(plan, OPS[op], dst, out, ld)
    back = from_dev(out).reshape(R, ld)
    assert np.array_equal(back[:, :Cc], logical)
    assert np.all(back[:, Cc:] == 0x1234)


# (workload, tensor, stored-transpose, operand, gemm)
WORKLOAD_OPERANDS = [
    ("tiny", "A", 0, "A", "tiny"),
    ("tiny", "B", 0, "B", "tiny"),
    ("qwen_fwd", "X", 0, "A", "qwen_gate_up"),
    ("qwen_fwd", "W_gate_up", 0, "B", "qwen_gate_up"),
    ("qwen_bwd", "H", 1, "A", "qwen_dW_down"),
    ("qwen_bwd", "dY", 0, "B", "qwen_dW_down"),
    ("qwen_bwd", "dY", 0, "A", "qwen_dH"),
    ("qwen_bwd", "W_down", 1, "B", "qwen_dH"),
]


@pytest.mark.parametrize("wl,tensor,trans,op,gemm", WORKLOAD_OPERANDS)
def test_pack_unpack_workload_operands(wl, tensor, trans, op, gemm):
    _, g = W.gemm_by_name(gemm)
    stored = W.draw(W.WORKLOADS[wl].tensors[tensor])
    plan, dst, logical = _check_pack(stored, trans, op, g.M, g.N, g.K, g.chiplets, g.grids[0], g.pages[0])
    _check_unpack(plan, op, dst, logical)


@pytest.mark.parametrize("gemm,tensor,trans,op,grid", [
    ("llama_up", "W_up", 0, "B", 2),
    ("llama_down", "W_down", 0, "B", 2),
    ("llama_dW_up", "X", 1, "A", 1),
    ("llama_dX", "W_up", 1, "B", 8),
    ("llama_dX", "W_up", 1, "B", 2),
])
def test_pack_llama_operands_full_size(gemm, tensor, trans, op, grid):
    wl, g = W.gemm_by_name(gemm)
    stored = W.draw(wl.tensors[tensor])
    plan, dst, logical = _check_pack(stored, trans, op, g.M, g.N, g.K, g.chiplets, grid, 4096)
    if not trans:
        _check_unpack(plan, op, dst, logical)


@pytest.mark.parametrize("M,N,K,G,Gr,P,op,trans,ld_extra", [
    (256, 512, 256, 4, 2, 2 * 1024 * 1024, "A", 0, 0),     # 64x padded strips
    (256, 512, 256, 4, 2, 65536, "B", 0, 8),                # padded strips, wider ld
    (256, 512, 256, 4, 2, 4096, "C", 0, 3),                 # ld not a multiple of 8: scalar path
    (384, 768, 201, 3, 1, 2048, "A", 0, 0),                 # 67-element slices: scalar path
    (384, 768, 201, 3, 1, 2048, "A", 1, 5),                 # transposed, ragged blocks
    (384, 768, 201, 3, 1, 128, "B", 1, 0),
    (256, 256, 512, 1, 1, 4096, "A", 1, 0),                 # single chiplet
    (1024, 256, 320, 8, 8, 4096, "B", 0, 0),                # 8x1 grid: K split in 40-row blocks
    (256, 1024, 512, 8, 1, 4096, "A", 1, 16),               # 1x8, transposed, wide ld
    (256, 256, 640, 2, 1, 4096, "A", 1, 8),                 # transposed: 10 register blocks per
                                                            # row, the last workgroup half idle
    (1024, 256, 2048, 8, 8, 4096, "B", 1, 0),               # transposed, 8x1: 256-row blocks
])
def test_pack_unpack_edge_cases(M, N, K, G, Gr, P, op, trans, ld_extra):
    R, Cc = OL.operand_shape(op, M, N, K)
    stored_shape = (Cc, R) if trans else (R, Cc)
    stored = W.draw_array(77 + R + Cc, *stored_shape, "normal", 1.0)
    ld = stored_shape[1] + ld_extra
    plan, dst, logical = _check_pack(stored, trans, op, M, N, K, G, Gr, P, ld=ld)
    _check_unpack(plan, op, dst, logical, ld=Cc + ld_extra)
