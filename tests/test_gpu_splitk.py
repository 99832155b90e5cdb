"""GPU parity of the split-K GEMM (ccl_gemm_splitk) against the oracle.

Each tile's K steps are cut into ranges whose fp32 partials are summed by a
second kernel; the result must meet the same bars as ccl_gemm_scaled:
relative Frobenius <= 5e-3 and max abs <= 1e-2 max|ref| for a bf16 C,
relative Frobenius <= 1e-4 for an fp32 C (only the fp32 summation order
differs from the fp64 oracle), and bit-exact on integer inputs, where the
split and unsplit GEMMs must also agree bit for bit. The workspace starts
filled with NaN bytes: its contents on entry must not matter.
"""
import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from paper_2606_11718_amd import ccl
from tests.helpers import torch_mod

pytestmark = pytest.mark.gpu

BF16, FP8, FP32 = ccl.CCL_DT_BF16, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_FP32


def _to_dev(a: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1)).to("cuda")


def _dev_bytes(n: int, value: int = 0xA5):
    torch = torch_mod()
    return torch.full((max(n, 1),), value, dtype=torch.uint8, device="cuda")


def _from_dev(t, dtype):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy().view(dtype)


def _draw(ab, seed, rows, cols, dist="normal", scale=1.0):
    if ab == FP8:
        return W.draw_array_fp8(seed, rows, cols, dist, scale)
    return W.draw_array(seed, rows, cols, dist, scale)


def _decode(ab, bits):
    return OG.decode_fp8_e4m3(bits) if ab == FP8 else OG.decode_bf16(bits)


def run_splitk(A, B, M, N, K, G, Gr, ab, c, splits, alpha=1.0, beta=0.0, C0=None,
               a_trans=0, b_trans=0, ws=None):
    """A, B as stored (transposed when *_trans). Returns the row-major C as
    float64 and the number of K ranges used."""
    plan = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ab, c)
    gr, gc = ccl.ccl_plan_grid(plan)
    ranges, need = ccl.ccl_gemm_splitk_workspace(plan, splits)
    print(f"splitk {M}x{N}x{K} grid {gr}x{gc} ab={ab} c={c} splits={splits} -> {ranges} "
          f"ws={need} alpha={alpha} beta={beta}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ac, Bc = _dev_bytes(la.total_bytes), _dev_bytes(lb.total_bytes)
    ccl.ccl_pack(plan, ccl.CCL_A, _to_dev(A), A.shape[1], a_trans, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, _to_dev(B), B.shape[1], b_trans, Bc)
    cdt = np.uint32 if c == FP32 else np.uint16
    Cc = _dev_bytes(lc.total_bytes) if C0 is None else _to_dev(OL.pack(C0.astype(cdt), gr, gc, 4096))
    if ws is None:
        ws = _dev_bytes(need, 0xFF)
    assert ws.numel() >= need
    # splits == 0 lets the library choose; the GEMM call takes the count it reported
    ccl.ccl_gemm_splitk(plan, alpha, Ac, Bc, beta, Cc, splits or ranges, ws, ws.numel())
    bits = OL.unpack(_from_dev(Cc, cdt), M, N, gr, gc, 4096)
    C = bits.view(np.float32).astype(np.float64) if c == FP32 else OG.decode_bf16(bits)
    return C, ranges


def _logical(stored, trans):
    return np.ascontiguousarray(stored.T) if trans else stored


@pytest.mark.parametrize("M,N,K,G,Gr,ta,tb,splits,ranges", [
    (768, 2048, 4096, 8, 1, 1, 0, 0, 2),       # Qwen3 dW_down (A = H^T stored), library's choice
    (768, 2048, 4096, 8, 1, 1, 0, 5, 5),       # 128 K steps in ranges of 26 (last one 24)
    (2048, 1536, 4096, 8, 2, 1, 0, 3, 3),      # Qwen3 dW_gate/up shape
    (4096, 768, 2048, 8, 8, 0, 1, 2, 2),       # B stored transposed
    (256, 512, 160, 1, 1, 0, 0, 4, 3),         # 5 K steps in ranges of 2: 2, 2, 1
    (256, 512, 160, 1, 1, 0, 0, 16, 5),        # one K step per range
    (1024, 1024, 16384, 8, 2, 0, 0, 16, 16),   # long K
])
@pytest.mark.parametrize("c", [BF16, FP32])
def test_splitk_bf16_matches_oracle(M, N, K, G, Gr, ta, tb, splits, ranges, c):
    A = _draw(BF16, 9100 + M + K, *((K, M) if ta else (M, K)))
    B = _draw(BF16, 9200 + N + K, *((N, K) if tb else (K, N)), "normal", 0.05)
    C, got_ranges = run_splitk(A, B, M, N, K, G, Gr, BF16, c, splits, a_trans=ta, b_trans=tb)
    assert got_ranges == ranges
    err = OG.errors(C, OG.gemm_fp64(_logical(A, ta), _logical(B, tb)))
    print("errors", err, flush=True)
    if c == FP32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


@pytest.mark.parametrize("tile,waves,M,N,K,G,Gr,splits", [
    ("128x128", 8, 768, 2048, 4096, 8, 1, 2),   # Qwen3 dW_down shape, 8 waves of 64x32
    ("256x128", 8, 2048, 1536, 4096, 8, 2, 3),  # 8 waves of 128x32
    ("128x256", 8, 1024, 2048, 2048, 8, 2, 4),
])
def test_splitk_eight_wave_tiles(tile, waves, M, N, K, G, Gr, splits, monkeypatch):
    monkeypatch.setenv("CCL_GEMM_TILE", tile)
    monkeypatch.setenv("CCL_GEMM_WAVES", str(waves))
    A = _draw(BF16, 9300 + M + K, M, K)
    B = _draw(BF16, 9400 + N + K, K, N, "normal", 0.05)
    C, got = run_splitk(A, B, M, N, K, G, Gr, BF16, FP32, splits)
    assert got == splits
    err = OG.errors(C, OG.gemm_fp64(A, B))
    print(tile, waves, "errors", err, flush=True)
    assert err["rel_fro"] <= 1e-4


@pytest.mark.parametrize("M,N,K,G,Gr,splits", [
    (768, 2048, 4096, 8, 1, 4),
    (256, 512, 320, 1, 1, 4),                  # 5 fp8 K steps: ranges 2, 2, 1
    (1024, 2048, 1024, 8, 2, 2),
])
@pytest.mark.parametrize("c", [BF16, FP32])
def test_splitk_fp8_matches_oracle(M, N, K, G, Gr, splits, c):
    A = _draw(FP8, 9300 + M + K, M, K)
    B = _draw(FP8, 9400 + N + K, K, N)
    C, _ = run_splitk(A, B, M, N, K, G, Gr, FP8, c, splits)
    err = OG.errors(C, OG.gemm_fp64(_decode(FP8, A), _decode(FP8, B)))
    print("errors", err, flush=True)
    if c == FP32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


@pytest.mark.parametrize("ab,c,alpha,beta", [(BF16, BF16, 1.5, -0.5), (BF16, FP32, 0.5, -1.0),
                                             (FP8, FP32, -2.0, 0.25)])
def test_splitk_scaled_matches_oracle(ab, c, alpha, beta):
    M, N, K, G, Gr = 768, 2048, 4096, 8, 1
    A = _draw(ab, 9500, M, K)
    B = _draw(ab, 9501, K, N, "normal", 0.05 if ab == BF16 else 1.0)
    if c == FP32:
        C0 = np.random.default_rng(9502).standard_normal((M, N)).astype(np.float32)
        C0_bits, C0_val = C0.view(np.uint32), C0.astype(np.float64)
    else:
        C0_bits = W.draw_array(9502, M, N, "normal", 2.0)
        C0_val = OG.decode_bf16(C0_bits)
    C, _ = run_splitk(A, B, M, N, K, G, Gr, ab, c, 4, alpha, beta, C0_bits)
    ref = OG.gemm_scaled_fp64(_decode(ab, A), _decode(ab, B), C0_val, alpha, beta)
    err = OG.errors(C, ref)
    print("errors", err, flush=True)
    if c == FP32:
        assert err["rel_fro"] <= 1e-4
    else:
        assert OG.within_tolerance(err)


@pytest.mark.parametrize("ab", [BF16, FP8])
def test_splitk_integer_inputs_bit_exact_and_equal_to_unsplit(ab):
    """Ternary inputs: every partial and every sum is an exact integer in
    fp32, so any range count gives the exact product."""
    M, N, K, G, Gr = 768, 2048, 4096, 8, 1
    A = _draw(ab, 9600, M, K, "ternary")
    B = _draw(ab, 9601, K, N, "ternary")
    exact = OG.gemm_fp64(_decode(ab, A), _decode(ab, B))
    assert np.abs(exact).max() < 2 ** 24
    outs = [run_splitk(A, B, M, N, K, G, Gr, ab, FP32, s)[0] for s in (1, 2, 7, 16)]
    for C in outs:
        assert np.array_equal(C, exact)


def test_splitk_beta_zero_does_not_read_c():
    M, N, K, G, Gr = 768, 2048, 4096, 8, 1
    A = _draw(BF16, 9700, M, K, "ternary")
    B = _draw(BF16, 9701, K, N, "ternary")
    nan_c = np.full((M, N), 0x7FC0, dtype=np.uint16)           # bf16 NaN everywhere
    C, _ = run_splitk(A, B, M, N, K, G, Gr, BF16, BF16, 4, -0.5, 0.0, nan_c)
    want = OG.decode_bf16(W.round_to_bf16_bits((-0.5 * OG.gemm_fp64(A, B)).astype(np.float32)))
    assert np.array_equal(C, want)


def test_one_workspace_serves_successive_gemms():
    """A workspace sized for the larger GEMM, reused in order on one stream
    by a smaller one: each result matches its own oracle."""
    big = (768, 2048, 4096, 8, 1)
    small = (256, 512, 1024, 4, 2)
    plan = ccl.ccl_plan(*big, 4096)
    _, need = ccl.ccl_gemm_splitk_workspace(plan, 8)
    ws = _dev_bytes(need, 0xFF)
    for i, (M, N, K, G, Gr) in enumerate((big, small)):
        A = _draw(BF16, 9800 + i, M, K)
        B = _draw(BF16, 9810 + i, K, N, "normal", 0.05)
        C, _ = run_splitk(A, B, M, N, K, G, Gr, BF16, FP32, 8, ws=ws)
        err = OG.errors(C, OG.gemm_fp64(A, B))
        print("errors", err, flush=True)
        assert err["rel_fro"] <= 1e-4


@pytest.mark.parametrize("M,N,K,G,Gr,splits", [
    (768, 2048, 4096, 8, 1, 2),     # 64-K ranges of 32 steps (rounds path)
    (768, 2048, 4096, 8, 1, 4),     # 16 steps per range
    (768, 2048, 4096, 8, 1, 5),     # 13 steps per range: per-step path
    (768, 2048, 4096, 8, 1, 3),     # 32-K ranges of 43 steps: not even, 32-K kernel
    (4096, 768, 2048, 8, 8, 2),
])
def test_splitk_k64_stages_equal_k32_bit_for_bit(M, N, K, G, Gr, splits, monkeypatch):
    """Where the K ranges are whole 64-K stages, the 64-K stage kernel
    writes the same partials as the 32-K one (same 32-K MFMA steps, same
    order), so the reduced C is identical bit for bit."""
    A = _draw(BF16, 9500 + M + K, M, K)
    B = _draw(BF16, 9600 + N + K, K, N, "normal", 0.05)
    C64, r64 = run_splitk(A, B, M, N, K, G, Gr, BF16, FP32, splits)
    monkeypatch.setenv("CCL_GEMM_STAGE_K", "32")
    C32, r32 = run_splitk(A, B, M, N, K, G, Gr, BF16, FP32, splits)
    assert r64 == r32 == splits
    assert np.array_equal(C64, C32)
    assert OG.errors(C64, OG.gemm_fp64(A, B))["rel_fro"] <= 1e-4
