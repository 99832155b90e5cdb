"""GPU parity of the CCL-native epilogue and of GEMM chaining in CCL.

  * ccl_gemm_scaled: C = alpha A B + beta C (the BLAS form of Sec. II-B)
    against the oracle's fp64 alpha A B + beta C, with the GEMM tolerance
    (relative Frobenius <= 5e-3, max abs <= 1e-2 max|ref|); bit-exact on
    integer inputs with power-of-two scalars; beta = 0 never reads C.
  * An FFN-style chain: the first GEMM's CCL output is the second GEMM's CCL
    A operand with no repack (the layouts are the same bytes), checked
    against the oracle's two fp64 GEMMs with the intermediate rounded to bf16.
"""
import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import compare_in_row_blocks, dev_full, from_dev, to_dev

pytestmark = pytest.mark.gpu


def _scaled(A, B, C0, M, N, K, G, Gr, P, alpha, beta, c_dev=None):
    """Pack A, B and C0 (row-major bf16 bits) and run ccl_gemm_scaled.
    Returns the row-major result bits (oracle unpack)."""
    plan = ccl.ccl_plan(M, N, K, G, Gr, P)
    gr, gc = ccl.ccl_plan_grid(plan)
    print(f"gemm_scaled {M}x{N}x{K} grid {gr}x{gc} alpha={alpha} beta={beta}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc = dev_full(la.total_bytes // 2), dev_full(lb.total_bytes // 2)
    ccl.ccl_pack(plan, ccl.CCL_A, to_dev(A), K, 0, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, to_dev(B), N, 0, Bc)
    if c_dev is None:
        c_dev = to_dev(OL.pack(C0, gr, gc, P))
    ccl.ccl_gemm_scaled(plan, alpha, Ac, Bc, beta, c_dev)
    return OL.unpack(from_dev(c_dev), M, N, gr, gc, P)


@pytest.mark.parametrize("M,N,K,G,Gr", [(256, 512, 256, 4, 2), (4096, 1536, 2048, 8, 2),
                                        (1024, 768, 1024, 8, 8)])
@pytest.mark.parametrize("alpha,beta", [(1.5, -0.5), (-1.0, 1.0), (0.25, 3.0)])
def test_scaled_matches_oracle(M, N, K, G, Gr, alpha, beta):
    A = W.draw_array(5100 + M, M, K, "normal", 1.0)
    B = W.draw_array(5200 + N, K, N, "normal", 0.05)
    C0 = W.draw_array(5300 + K, M, N, "normal", 2.0)
    got = _scaled(A, B, C0, M, N, K, G, Gr, 4096, alpha, beta)
    ref = OG.gemm_scaled_fp64(A, B, C0, alpha, beta)
    err = OG.errors(OG.decode_bf16(got), ref)
    print("errors", err, flush=True)
    assert OG.within_tolerance(err)


@pytest.mark.parametrize("alpha,beta", [(1.0, -1.0), (0.5, 2.0), (-2.0, 0.25)])
def test_scaled_integer_inputs_bit_exact(alpha, beta):
    """Ternary A, B, C and power-of-two scalars: alpha*acc + beta*c is exact
    in fp32, so the bf16 result is the round-to-nearest-even of the exact
    value."""
    M, N, K, G, Gr = 512, 1024, 256, 8, 2
    A = W.draw_array(61, M, K, "ternary")
    B = W.draw_array(62, K, N, "ternary")
    C0 = W.draw_array(63, M, N, "ternary")
    exact = OG.gemm_scaled_fp64(A, B, C0, alpha, beta)
    assert np.abs(exact).max() < 2 ** 24
    want = W.round_to_bf16_bits(exact.astype(np.float32))
    got = _scaled(A, B, C0, M, N, K, G, Gr, 4096, alpha, beta)
    assert np.array_equal(got, want)


def test_beta_zero_does_not_read_c():
    M, N, K, G, Gr = 512, 512, 256, 4, 2
    A = W.draw_array(64, M, K, "ternary")
    B = W.draw_array(65, K, N, "ternary")
    plan = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    lc = ccl.ccl_plan_layout(plan, ccl.CCL_C)
    c_dev = dev_full(lc.total_bytes // 2, 0x7FC0)           # bf16 NaN everywhere
    got = _scaled(A, B, None, M, N, K, G, Gr, 4096, -0.5, 0.0, c_dev=c_dev)
    want = W.round_to_bf16_bits((-0.5 * OG.gemm_fp64(A, B)).astype(np.float32))
    assert np.array_equal(got, want)


def test_alpha_one_beta_zero_equals_ccl_gemm():
    M, N, K, G, Gr = 1024, 1024, 512, 8, 2
    A = W.draw_array(66, M, K, "normal", 1.0)
    B = W.draw_array(67, K, N, "normal", 0.05)
    plan = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc = dev_full(la.total_bytes // 2), dev_full(lb.total_bytes // 2)
    ccl.ccl_pack(plan, ccl.CCL_A, to_dev(A), K, 0, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, to_dev(B), N, 0, Bc)
    C1, C2 = dev_full(lc.total_bytes // 2), dev_full(lc.total_bytes // 2)
    ccl.ccl_gemm(plan, Ac, Bc, C1)
    ccl.ccl_gemm_scaled(plan, 1.0, Ac, Bc, 0.0, C2)
    assert np.array_equal(from_dev(C1), from_dev(C2))


def test_llama_up_scaled_full_compare():
    """alpha X W_up + beta C0 at the Llama-3.1-70B forward shape: every
    element against the oracle's fp64 alpha A B + beta C0, in row blocks."""
    wl, g = W.gemm_by_name("llama_up")
    X = W.draw(wl.tensors["X"])
    Wu = W.draw(wl.tensors["W_up"])
    C0 = W.draw_array(68, g.M, g.N, "normal", 1.0)
    alpha, beta = 0.5, -1.0
    plan = ccl.ccl_plan(g.M, g.N, g.K, 8, 2, 4096)
    gr, gc = ccl.ccl_plan_grid(plan)
    print(f"llama_up scaled grid {gr}x{gc}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc, Cc = (dev_full(l.total_bytes // 2) for l in (la, lb, lc))
    ccl.ccl_pack(plan, ccl.CCL_A, to_dev(X), g.K, 0, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, to_dev(Wu), g.N, 0, Bc)
    ccl.ccl_pack(plan, ccl.CCL_C, to_dev(C0), g.N, 0, Cc)
    ccl.ccl_gemm_scaled(plan, alpha, Ac, Bc, beta, Cc)
    cbuf = from_dev(Cc)
    del Ac, Bc, Cc
    Wu_d = OG.decode(Wu)
    err = compare_in_row_blocks(
        {0: (cbuf, gr, gc)}, g.M, g.N, 4096,
        lambda r0, r1: OG.gemm_scaled_fp64(OG.decode(X[r0:r1]), Wu_d, C0[r0:r1], alpha, beta),
        OG.decode_bf16)[0]
    print("errors over all of C", err, flush=True)
    assert OG.within_tolerance(err)


def test_ffn_chain_without_repack():
    """Y = (X W1) W2 with the intermediate kept in CCL: the first GEMM's C
    buffer is passed as the second GEMM's A buffer."""
    T, D, F, G, Gr, P = 2048, 1024, 3072, 8, 2, 4096
    X = W.draw_array(81, T, D, "normal", 1.0)
    W1 = W.draw_array(82, D, F, "normal", 0.03)
    W2 = W.draw_array(83, F, D, "normal", 0.02)
    up = ccl.ccl_plan(T, F, D, G, Gr, P)
    down = ccl.ccl_plan(T, D, F, G, Gr, P)
    assert ccl.ccl_plan_layout(up, ccl.CCL_C) == ccl.ccl_plan_layout(down, ccl.CCL_A)
    Xc = dev_full(ccl.ccl_plan_layout(up, ccl.CCL_A).total_bytes // 2)
    W1c = dev_full(ccl.ccl_plan_layout(up, ccl.CCL_B).total_bytes // 2)
    W2c = dev_full(ccl.ccl_plan_layout(down, ccl.CCL_B).total_bytes // 2)
    Hc = dev_full(ccl.ccl_plan_layout(up, ccl.CCL_C).total_bytes // 2)
    Yc = dev_full(ccl.ccl_plan_layout(down, ccl.CCL_C).total_bytes // 2)
    ccl.ccl_pack(up, ccl.CCL_A, to_dev(X), D, 0, Xc)
    ccl.ccl_pack(up, ccl.CCL_B, to_dev(W1), F, 0, W1c)
    ccl.ccl_pack(down, ccl.CCL_B, to_dev(W2), D, 0, W2c)
    ccl.ccl_gemm(up, Xc, W1c, Hc)
    ccl.ccl_gemm(down, Hc, W2c, Yc)
    Y = OL.unpack(from_dev(Yc), T, D, Gr, G // Gr, P)
    H_ref = W.round_to_bf16_bits(OG.gemm_fp64(X, W1).astype(np.float32))
    Y_ref = OG.gemm_fp64(H_ref, W2)
    err = OG.errors(OG.decode_bf16(Y), Y_ref)
    print("chain errors", err, flush=True)
    assert OG.within_tolerance(err)
