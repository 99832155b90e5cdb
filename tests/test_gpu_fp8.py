"""GPU parity of the fp8 (E4M3) GEMM on CCL operands (Fig. 7 data types).

The oracle decodes the same fp8 bits exactly and multiplies in fp64; the GPU
multiplies on the matrix cores with fp32 accumulation. Tolerances: the GEMM
bar (relative Frobenius <= 5e-3, max abs <= 1e-2 max|ref|) for a bf16 C;
relative Frobenius <= 1e-4 for an fp32 C (fp8 products are exact in fp32,
so only the summation order differs); bit-exact on integer inputs.
"""
import os

import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import compare_in_row_blocks, torch_mod

pytestmark = pytest.mark.gpu


def _to_dev(a: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1)).to("cuda")


def _dev_bytes(n: int, value: int = 0xA5):
    torch = torch_mod()
    return torch.full((n,), value, dtype=torch.uint8, device="cuda")


def _from_dev(t, dtype):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy().view(dtype)


def run_fp8(A, B, M, N, K, G, Gr, c_type=ccl.CCL_DT_BF16, tile=None, waves=None, alpha=1.0,
            beta=0.0, C0=None, a_trans=0, b_trans=0, unpack=True):
    """A, B: fp8 bits (uint8) as stored (transposed when *_trans). Returns C
    as float64 (oracle unpack of the GPU's CCL buffer; None when unpack is
    False) and the CCL buffer."""
    if tile:
        os.environ["CCL_GEMM_TILE"] = tile
    if waves:
        os.environ["CCL_GEMM_WAVES"] = str(waves)
    try:
        plan = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ccl.CCL_DT_FP8_E4M3, c_type)
    finally:
        os.environ.pop("CCL_GEMM_TILE", None)
        os.environ.pop("CCL_GEMM_WAVES", None)
    gr, gc = ccl.ccl_plan_grid(plan)
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(plan)
    print(f"fp8 gemm {M}x{N}x{K} grid {gr}x{gc} tile {tm_}x{tn_} wgs={wgs} c={c_type} "
          f"alpha={alpha} beta={beta}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc = _dev_bytes(la.total_bytes), _dev_bytes(lb.total_bytes)
    ccl.ccl_pack(plan, ccl.CCL_A, _to_dev(A), A.shape[1], a_trans, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, _to_dev(B), B.shape[1], b_trans, Bc)
    cdt = np.uint32 if c_type == ccl.CCL_DT_FP32 else np.uint16
    if C0 is None:
        Cc = _dev_bytes(lc.total_bytes)
    else:
        Cc = _to_dev(OL.pack(C0.astype(cdt), gr, gc, 4096))
    if alpha == 1.0 and beta == 0.0:
        ccl.ccl_gemm(plan, Ac, Bc, Cc)
    else:
        ccl.ccl_gemm_scaled(plan, alpha, Ac, Bc, beta, Cc)
    cbuf = _from_dev(Cc, cdt)
    if not unpack:
        return None, cbuf, (gr, gc)
    Cbits = OL.unpack(cbuf, M, N, gr, gc, 4096)
    C = Cbits.view(np.float32).astype(np.float64) if cdt == np.uint32 else OG.decode_bf16(Cbits)
    return C, cbuf, (gr, gc)


def _logical(stored, trans):
    return np.ascontiguousarray(stored.T) if trans else stored


@pytest.mark.parametrize("M,N,K,G,Gr,ta,tb", [
    (256, 512, 256, 4, 2, 0, 0),                 # tiny shape
    (4096, 1536, 2048, 8, 2, 0, 0),              # Qwen3 gate/up forward shape
    (768, 2048, 4096, 8, 1, 1, 0),               # Qwen3 dW_down shape (A stored transposed)
    (4096, 768, 2048, 8, 8, 0, 1),               # Qwen3 dH shape (B stored transposed)
    (1024, 1024, 576, 1, 1, 0, 0),               # 9 K steps: ragged against the 4-stage loop
    (128, 128, 64, 1, 1, 0, 0),                  # one tile, one K step
    (1024, 1024, 640, 1, 1, 0, 0),               # 16x16x128 kernel: 5 steps of 128 (odd)
    (2048, 2048, 1024, 8, 2, 1, 1),              # 16x16x128 kernel: both stored transposed,
                                                 # K blocks of 2 (A) and 4 (B) steps
])
@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_fp8_gemm_matches_oracle(M, N, K, G, Gr, ta, tb, c_type):
    A = W.draw_array_fp8(8100 + M + K, *((K, M) if ta else (M, K)), "normal", 1.0)
    B = W.draw_array_fp8(8200 + N + K, *((N, K) if tb else (K, N)), "normal", 1.0)
    C, _, _ = run_fp8(A, B, M, N, K, G, Gr, c_type, a_trans=ta, b_trans=tb)
    err = OG.errors(C, OG.gemm_fp64(_logical(A, ta), _logical(B, tb)))
    print("errors", err, flush=True)
    if c_type == ccl.CCL_DT_FP32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


@pytest.mark.parametrize("tile,waves,M,N,K,G,Gr", [
    ("256x256", 8, 1024, 2048, 1024, 8, 2),
    ("256x256", 4, 1024, 2048, 1024, 8, 2),
    ("256x128", 4, 1024, 2048, 1024, 8, 2),
    ("128x256", 4, 1024, 2048, 1024, 8, 2),
    ("128x128", 4, 1024, 2048, 1024, 8, 2),
    ("128x128", 4, 512, 1024, 1088, 1, 1),       # 17 K steps
])
def test_fp8_every_kernel_variant(tile, waves, M, N, K, G, Gr):
    A = W.draw_array_fp8(8300 + M, M, K, "normal", 1.0)
    B = W.draw_array_fp8(8400 + N, K, N, "normal", 1.0)
    C, _, _ = run_fp8(A, B, M, N, K, G, Gr, ccl.CCL_DT_FP32, tile=tile, waves=waves)
    err = OG.errors(C, OG.gemm_fp64(A, B))
    print(tile, waves, "errors", err, flush=True)
    assert err["rel_fro"] <= 1e-4


@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_fp8_integer_inputs_bit_exact(c_type):
    M, N, K, G, Gr = 1024, 2048, 512, 8, 2
    A = W.draw_array_fp8(91, M, K, "ternary")
    B = W.draw_array_fp8(92, K, N, "ternary")
    ref = OG.gemm_fp64(A, B)
    assert np.abs(ref).max() <= 256
    C, _, _ = run_fp8(A, B, M, N, K, G, Gr, c_type)
    assert np.array_equal(C, ref)


def test_fp8_identity_returns_a():
    M, K = 512, 512
    A = W.draw_array_fp8(93, M, K, "normal", 4.0)
    I = W.round_to_fp8_e4m3_bits(np.eye(K, dtype=np.float32))
    C, _, _ = run_fp8(A, I, M, K, K, 4, 2, ccl.CCL_DT_FP32)
    assert np.array_equal(C, OG.decode_fp8_e4m3(A))


@pytest.mark.parametrize("alpha,beta", [(0.5, -1.0), (2.0, 0.25)])
def test_fp8_scaled_fp32_output(alpha, beta):
    M, N, K, G, Gr = 1024, 1024, 512, 8, 2
    A = W.draw_array_fp8(94, M, K, "normal", 1.0)
    B = W.draw_array_fp8(95, K, N, "normal", 1.0)
    C0 = np.random.default_rng(96).standard_normal((M, N)).astype(np.float32)
    C, _, _ = run_fp8(A, B, M, N, K, G, Gr, ccl.CCL_DT_FP32, alpha=alpha, beta=beta,
                      C0=C0.view(np.uint32))
    err = OG.errors(C, OG.gemm_scaled_fp64(A, B, C0.astype(np.float64), alpha, beta))
    print("errors", err, flush=True)
    assert err["rel_fro"] <= 1e-4


@pytest.mark.parametrize("name", ["llama_up", "llama_down"])
def test_fp8_llama_forward_full_compare(name):
    """fp8 X W_up / H W_down at the Llama-3.1-70B forward shape (fp32 C):
    every element against the fp64 oracle, in row blocks of 1024."""
    _, g = W.gemm_by_name(name)
    A = W.draw_array_fp8(8500 + g.K, g.M, g.K, "normal", 1.0)
    B = W.draw_array_fp8(8600 + g.N, g.K, g.N, "normal", 1.0)
    _, cbuf, (gr, gc) = run_fp8(A, B, g.M, g.N, g.K, 8, 2, ccl.CCL_DT_FP32, unpack=False)
    B_d = OG.decode(B)
    err = compare_in_row_blocks({0: (cbuf, gr, gc)}, g.M, g.N, 4096,
                                lambda r0, r1: OG.gemm_fp64(OG.decode(A[r0:r1]), B_d),
                                lambda bits: bits.view(np.float32).astype(np.float64))[0]
    print(name, "errors over all of C", err, flush=True)
    assert err["rel_fro"] <= 1e-4
    assert err["max_abs"] <= 1e-2 * err["max_ref"]


@pytest.mark.parametrize("remap", [0, 1])
@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_fp8_rowmajor_baseline(remap, c_type):
    """The same fp8 kernel on plain row-major operands (the layout the paper
    starts from), with the native or the XCD-aware tile map."""
    M, N, K, G, Gr = 1024, 2048, 1024, 8, 2
    A = W.draw_array_fp8(97, M, K, "normal", 1.0)
    B = W.draw_array_fp8(98, K, N, "normal", 1.0)
    plan = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ccl.CCL_DT_FP8_E4M3, c_type)
    e = 4 if c_type == ccl.CCL_DT_FP32 else 2
    print(f"fp8 rowmajor {M}x{N}x{K} remap={remap} c_bytes={e}", flush=True)
    Cd = _dev_bytes(M * N * e)
    ccl.ccl_gemm_rowmajor(plan, _to_dev(A), _to_dev(B), Cd, remap)
    Cb = _from_dev(Cd, np.uint32 if e == 4 else np.uint16).reshape(M, N)
    C = Cb.view(np.float32).astype(np.float64) if e == 4 else OG.decode_bf16(Cb)
    err = OG.errors(C, OG.gemm_fp64(A, B))
    print("errors", err, flush=True)
    if e == 4:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


def _run_pipe(on, A, B, M, N, K, G, Gr, c_type):
    os.environ["CCL_GEMM_FP8_PIPE"] = "1" if on else "0"
    try:
        _, cbuf, grid = run_fp8(A, B, M, N, K, G, Gr, c_type, tile="256x256", waves=8, unpack=False)
    finally:
        os.environ.pop("CCL_GEMM_FP8_PIPE", None)
    return cbuf, grid


@pytest.mark.parametrize("M,N,K,G,Gr", [(512, 512, 128 * s, 1, 1)
                                        for s in (1, 2, 3, 4, 5, 6, 7, 8, 11, 13, 14, 19, 20)]
                         + [(2048, 2048, 1024, 8, 2), (2048, 2048, 2048, 8, 1), (2048, 2048, 2048, 8, 8)])
@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_fp8_pipelined_equals_two_stage_bit_for_bit(M, N, K, G, Gr, c_type):
    """The pipelined 16x16x128 kernel issues every accumulator's MFMAs in the
    same K order as the two-stage one, so C is identical bit for bit: for
    step counts that stop inside the prologue, the tail alone (up to 7
    steps), one or more groups of six steps with tails of 0 to 7, and over
    CCL K blocks of 2 and 4 steps; and within the oracle's tolerance."""
    A = W.draw_array_fp8(8700 + K + Gr, M, K, "normal", 1.0)
    B = W.draw_array_fp8(8800 + K + Gr, K, N, "normal", 1.0)
    on, (gr, gc) = _run_pipe(True, A, B, M, N, K, G, Gr, c_type)
    off, _ = _run_pipe(False, A, B, M, N, K, G, Gr, c_type)
    assert np.array_equal(on, off)
    bits = OL.unpack(on, M, N, gr, gc, 4096)
    C = bits.view(np.float32).astype(np.float64) if c_type == ccl.CCL_DT_FP32 else OG.decode_bf16(bits)
    err = OG.errors(C, OG.gemm_fp64(A, B))
    print("errors", err, flush=True)
    if c_type == ccl.CCL_DT_FP32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)
