"""GPU parity for the other element types (Fig. 7 data types).

  * ccl_pack / ccl_unpack of 1-byte (fp8 E4M3) and 4-byte (fp32) operands
    against the oracle's CCL map, bit-exact, on the 16-byte vector path and
    the per-element path, row-major and stored-transpose sources, padding
    left untouched;
  * ccl_gemm / ccl_gemm_scaled with an fp32 C on bf16 operands against the
    oracle's fp64 product (GEMM tolerance), and bit-exact on integer inputs.
"""
import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import to_dev, torch_mod

pytestmark = pytest.mark.gpu

OPS = {"A": ccl.CCL_A, "B": ccl.CCL_B, "C": ccl.CCL_C}
DT = {1: ccl.CCL_DT_FP8_E4M3, 2: ccl.CCL_DT_BF16, 4: ccl.CCL_DT_FP32}
NP = {1: np.uint8, 2: np.uint16, 4: np.uint32}
FILL = 0xA5


def bytes_to_dev(a: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1)).to("cuda")


def dev_bytes(n: int, value: int = FILL):
    torch = torch_mod()
    return torch.full((n,), value, dtype=torch.uint8, device="cuda")


def dev_to(t, dtype) -> np.ndarray:
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy().view(dtype)


def _bits(seed, rows, cols, e):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 1 << (8 * e), size=(rows, cols), dtype=np.uint64).astype(NP[e])


CASES = [
    # M, N, K, G, Gr, P, op, trans, e_ab, e_c, ld_pad
    (256, 512, 256, 4, 2, 4096, "A", 0, 1, 2, 0),        # fp8 vector path
    (256, 512, 256, 4, 2, 4096, "B", 1, 1, 2, 0),        # fp8 from the stored transpose (tiled)
    (256, 512, 256, 4, 2, 4096, "C", 0, 1, 4, 0),        # fp32 C
    (512, 256, 192, 4, 4, 65536, "A", 1, 1, 4, 16),      # fp8, padded strips, ld > rows
    (384, 768, 201, 3, 1, 2048, "A", 0, 1, 2, 3),        # fp8 per-element path (odd widths)
    (384, 768, 201, 3, 1, 2048, "B", 1, 1, 2, 5),        # fp8 transpose, per-element path
    (384, 768, 201, 3, 1, 2048, "C", 0, 2, 4, 1),        # fp32 C, per-element path
    (1024, 2048, 512, 8, 2, 4096, "C", 0, 2, 4, 0),      # fp32 C, 8 chiplets
    (256, 1024, 512, 8, 1, 4096, "B", 0, 1, 4, 0),       # fp8 B, 1 x 8
    (256, 256, 1280, 2, 1, 4096, "A", 1, 1, 2, 16),      # fp8 transpose, register blocks:
                                                          # 10 blocks per row, 4 per workgroup
    (256, 512, 256, 4, 2, 4096, "B", 1, 4, 4, 4),        # fp32 A/B plan, transpose (32x32 blocks)
    (512, 256, 192, 4, 4, 4096, "A", 1, 4, 4, 0),        # fp32 transpose, 6 blocks per strip row
]


@pytest.mark.parametrize("M,N,K,G,Gr,P,op,trans,eab,ec,ldpad", CASES)
def test_typed_pack_unpack(M, N, K, G, Gr, P, op, trans, eab, ec, ldpad):
    plan = ccl.ccl_plan_typed(M, N, K, G, Gr, P, DT[eab], DT[ec])
    gr, gc = ccl.ccl_plan_grid(plan)
    lay = ccl.ccl_plan_layout(plan, OPS[op])
    e = lay.elem_bytes
    R, Cc = OL.operand_shape(op, M, N, K)
    logical = _bits(7000 + M + K + e, R, Cc, e)
    stored = np.ascontiguousarray(logical.T) if trans else logical
    ld = stored.shape[1] + ldpad
    src = np.zeros((stored.shape[0], ld), dtype=NP[e])
    src[:, :stored.shape[1]] = stored
    print(f"typed pack {op} {R}x{Cc} e={e} grid {gr}x{gc} P={P} trans={trans} ld={ld}", flush=True)
    dst = dev_bytes(lay.total_bytes)
    ccl.ccl_pack(plan, OPS[op], bytes_to_dev(src), ld, trans, dst)
    got = dev_to(dst, NP[e])
    ref = OL.pack_reshape(logical, gr, gc, P)
    pad = OL.padding_mask(R, Cc, gr, gc, P, e)
    assert np.array_equal(got[~pad], ref[~pad])
    assert np.all(got.view(np.uint8).reshape(-1, e)[pad] == FILL)
    if not trans:
        out = dev_bytes(R * ld * e, 0x3C)
        ccl.ccl_unpack(plan, OPS[op], dst, out, ld)
        back = dev_to(out, NP[e]).reshape(R, ld)
        assert np.array_equal(back[:, :Cc], logical)
        assert np.all(back[:, Cc:].view(np.uint8) == 0x3C)


def _gemm_f32(A, B, M, N, K, G, Gr, alpha=1.0, beta=0.0, C0=None):
    plan = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ccl.CCL_DT_BF16, ccl.CCL_DT_FP32)
    gr, gc = ccl.ccl_plan_grid(plan)
    print(f"gemm fp32-C {M}x{N}x{K} grid {gr}x{gc} alpha={alpha} beta={beta}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    assert lc.elem_bytes == 4
    Ac, Bc = dev_bytes(la.total_bytes), dev_bytes(lb.total_bytes)
    ccl.ccl_pack(plan, ccl.CCL_A, to_dev(A), K, 0, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, to_dev(B), N, 0, Bc)
    if C0 is None:
        Cc = dev_bytes(lc.total_bytes)
    else:
        Cc = bytes_to_dev(OL.pack(np.ascontiguousarray(C0, dtype=np.float32).view(np.uint32), gr, gc, 4096))
    if alpha == 1.0 and beta == 0.0:
        ccl.ccl_gemm(plan, Ac, Bc, Cc)
    else:
        ccl.ccl_gemm_scaled(plan, alpha, Ac, Bc, beta, Cc)
    bits = OL.unpack(dev_to(Cc, np.uint32), M, N, gr, gc, 4096)
    return bits.view(np.float32).astype(np.float64)


@pytest.mark.parametrize("M,N,K,G,Gr", [(256, 512, 256, 4, 2), (4096, 1536, 2048, 8, 2),
                                        (768, 2048, 4096, 8, 1)])
def test_gemm_fp32_output_matches_oracle(M, N, K, G, Gr):
    A = W.draw_array(7100 + M, M, K, "normal", 1.0)
    B = W.draw_array(7200 + N, K, N, "normal", 0.05)
    got = _gemm_f32(A, B, M, N, K, G, Gr)
    err = OG.errors(got, OG.gemm_fp64(A, B))
    print("errors", err, flush=True)
    # fp32 output: only the fp32 accumulation order differs from the fp64 sum
    assert err["rel_fro"] <= 1e-4


def test_gemm_fp32_output_integer_exact():
    M, N, K, G, Gr = 512, 1024, 512, 8, 2
    A = W.draw_array(73, M, K, "ternary")
    B = W.draw_array(74, K, N, "ternary")
    got = _gemm_f32(A, B, M, N, K, G, Gr)
    assert np.array_equal(got, OG.gemm_fp64(A, B))


@pytest.mark.parametrize("alpha,beta", [(0.5, -2.0), (-1.5, 0.25)])
def test_gemm_scaled_fp32_output(alpha, beta):
    M, N, K, G, Gr = 1024, 1024, 512, 8, 2
    A = W.draw_array(75, M, K, "normal", 1.0)
    B = W.draw_array(76, K, N, "normal", 0.05)
    C0 = np.random.default_rng(77).standard_normal((M, N)).astype(np.float32)
    got = _gemm_f32(A, B, M, N, K, G, Gr, alpha, beta, C0)
    ref = OG.gemm_scaled_fp64(A, B, C0.astype(np.float64), alpha, beta)
    err = OG.errors(got, ref)
    print("errors", err, flush=True)
    assert err["rel_fro"] <= 1e-4
