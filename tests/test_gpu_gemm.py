"""GPU parity of ccl_gemm with the fp64 oracle (Sec. II-B C = A B).

Tolerance: relative Frobenius error <= 5e-3 and max abs error <= 1e-2 *
max|C_ref|. C is read back through the oracle's own unpack of the GPU's CCL
buffer and every element is compared; the Llama-sized products are
compared in row blocks (the oracle's fp64 rows computed once per block).
Integer-valued cases are bit-exact.
"""
import os

import numpy as np
import pytest

import workloads as W
from oracle import gemm as OG
from oracle import layout as OL
from oracle import plan as OP
from paper_2606_11718_amd import ccl
from tests.helpers import CANARY, compare_in_row_blocks, dev_full, from_dev, to_dev

pytestmark = pytest.mark.gpu


def run_gemm(A_stored, a_trans, B_stored, b_trans, M, N, K, G, Gr, P, tile=None, unpack=True,
             waves=None):
    """Pack A and B on the GPU and run the GEMM. Returns (C, plan) where C is
    the row-major bf16 bits (oracle unpack), or (ccl buffer, Gr, Gc) when
    unpack is False. tile / waves force the kernel variant."""
    if tile:
        os.environ["CCL_GEMM_TILE"] = tile
    if waves:
        os.environ["CCL_GEMM_WAVES"] = str(waves)
    try:
        plan = ccl.ccl_plan(M, N, K, G, Gr, P)
    finally:
        os.environ.pop("CCL_GEMM_TILE", None)
        os.environ.pop("CCL_GEMM_WAVES", None)
    gr, gc = ccl.ccl_plan_grid(plan)
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(plan)
    print(f"gemm {M}x{N}x{K} grid {gr}x{gc} P={P} tile {tm_}x{tn_} wgs={wgs} "
          f"trans=({a_trans},{b_trans})", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    Ad, Bd = to_dev(A_stored), to_dev(B_stored)
    Ac, Bc, Cc = dev_full(la.total_bytes // 2), dev_full(lb.total_bytes // 2), dev_full(lc.total_bytes // 2)
    ccl.ccl_pack(plan, ccl.CCL_A, Ad, A_stored.shape[1], a_trans, Ac)
    ccl.ccl_pack(plan, ccl.CCL_B, Bd, B_stored.shape[1], b_trans, Bc)
    del Ad, Bd
    ccl.ccl_gemm(plan, Ac, Bc, Cc)
    cbuf = from_dev(Cc)
    if lc.total_bytes != lc.strip_bytes * gr * gc:       # padding untouched
        assert np.all(cbuf[OL.padding_mask(M, N, gr, gc, P)] == CANARY)
    return (OL.unpack(cbuf, M, N, gr, gc, P) if unpack else (cbuf, gr, gc)), plan


def _logical(stored, trans):
    return np.ascontiguousarray(stored.T) if trans else stored


def _check_full(A_stored, a_trans, B_stored, b_trans, M, N, K, G, Gr, P, tile=None, waves=None):
    Cbits, _ = run_gemm(A_stored, a_trans, B_stored, b_trans, M, N, K, G, Gr, P, tile, waves=waves)
    C_ref = OG.gemm_fp64(_logical(A_stored, a_trans), _logical(B_stored, b_trans))
    err = OG.errors(OG.decode_bf16(Cbits), C_ref)
    print("errors", err, flush=True)
    assert err["rel_fro"] <= 5e-3
    assert err["max_abs"] <= 1e-2 * err["max_ref"]
    return err


@pytest.mark.parametrize("gemm", ["tiny", "qwen_gate_up", "qwen_dW_down", "qwen_dH"])
def test_gemm_workloads_full_compare(gemm):
    wl, g = W.gemm_by_name(gemm)
    A = W.draw(wl.tensors[g.a_src])
    B = W.draw(wl.tensors[g.b_src])
    _check_full(A, g.a_trans, B, g.b_trans, g.M, g.N, g.K, g.chiplets, g.grids[0], g.pages[0])


def test_qwen_backward_grids_are_the_automatic_choice():
    for name, expect in (("qwen_dW_down", 1), ("qwen_dH", 8)):
        _, g = W.gemm_by_name(name)
        p = ccl.ccl_plan(g.M, g.N, g.K, g.chiplets, 0, 4096)
        assert ccl.ccl_plan_grid(p)[0] == expect == OP.auto_grid_rows(g.M, g.N, g.K, g.chiplets)


@pytest.mark.parametrize("tile,waves", [("256x256", 8), ("256x128", 4), ("128x256", 4),
                                        ("128x128", 4), ("256x128", 8), ("128x256", 8),
                                        ("128x128", 8)])
@pytest.mark.parametrize("M,N,K,G,Gr", [(2048, 2048, 1024, 8, 2),      # 2x4 grid, 32 K steps
                                        (1024, 1024, 1056, 1, 1)])     # 33 K steps: ragged stage ring
def test_gemm_every_kernel_variant(tile, waves, M, N, K, G, Gr):
    A = W.draw_array(901, M, K, "normal", 1.0)
    B = W.draw_array(902, K, N, "normal", 0.02)
    _check_full(A, 0, B, 0, M, N, K, G, Gr, 4096, tile, waves)


@pytest.mark.parametrize("tile", ["256x128", "128x256", "128x128"])
@pytest.mark.parametrize("steps", [1, 2, 3, 5, 7, 12, 13, 19, 28, 45])
def test_gemm_stage_ring_step_counts(tile, steps):
    """K step counts that stop inside the first lone step, the first
    rounds, the loop and the tail of the rounds path of the smaller tiles
    (one chiplet, so one K block per operand)."""
    M, N, K = 256, 256, 32 * steps
    A = W.draw_array(951 + steps, M, K, "normal", 1.0)
    B = W.draw_array(952 + steps, K, N, "normal", 0.05)
    _check_full(A, 0, B, 0, M, N, K, 1, 1, 4096, tile, 8)


def _run_stage_k(stage_k, A, B, M, N, K, G, Gr, tile):
    if stage_k == 32:
        os.environ["CCL_GEMM_STAGE_K"] = "32"
    try:
        Cbits, _ = run_gemm(A, 0, B, 0, M, N, K, G, Gr, 4096, tile, waves=8)
    finally:
        os.environ.pop("CCL_GEMM_STAGE_K", None)
    return Cbits


@pytest.mark.parametrize("tile", ["256x128", "128x256", "128x128"])
@pytest.mark.parametrize("M,N,K,G,Gr", [(4096, 1536, 2048, 8, 2),     # Qwen3 gate/up grid
                                        (768, 2048, 4096, 8, 1),      # dW_down grid (1x8)
                                        (4096, 768, 2048, 8, 8),      # dH grid (8x1)
                                        (1024, 1024, 1344, 1, 1)])    # one block, 21 stages
def test_gemm_k64_stages_equal_k32_bit_for_bit(tile, M, N, K, G, Gr):
    """The 64-K stage kernel adds the same 32-K MFMA steps in the same K
    order as the 32-K kernel, so C is identical bit for bit; and within
    the oracle's tolerance."""
    if (tile == "256x128" and (M // Gr) % 256) or (tile == "128x256" and (N // (G // Gr)) % 256):
        pytest.skip("tile does not divide the partition")
    A = W.draw_array(961, M, K, "normal", 1.0)
    B = W.draw_array(962, K, N, "normal", 0.02)
    c64 = _run_stage_k(64, A, B, M, N, K, G, Gr, tile)
    c32 = _run_stage_k(32, A, B, M, N, K, G, Gr, tile)
    assert np.array_equal(c64, c32)
    err = OG.errors(OG.decode_bf16(c64), OG.gemm_fp64(A, B))
    assert err["rel_fro"] <= 5e-3 and err["max_abs"] <= 1e-2 * err["max_ref"]


@pytest.mark.parametrize("tile", ["256x128", "128x256", "128x128"])
@pytest.mark.parametrize("stages", [1, 2, 3, 4, 5, 6, 7, 11, 13, 17, 25])
def test_gemm_k64_stage_counts(tile, stages):
    """64-K stage counts that stop inside the lone first steps, the rounds,
    the loop and the tail of the 3- and 4-stage rings (one chiplet: one K
    block per operand)."""
    M, N, K = 256, 256, 64 * stages
    A = W.draw_array(971 + stages, M, K, "normal", 1.0)
    B = W.draw_array(972 + stages, K, N, "normal", 0.05)
    c64 = _run_stage_k(64, A, B, M, N, K, 1, 1, tile)
    c32 = _run_stage_k(32, A, B, M, N, K, 1, 1, tile)
    assert np.array_equal(c64, c32)
    err = OG.errors(OG.decode_bf16(c64), OG.gemm_fp64(A, B))
    assert err["rel_fro"] <= 5e-3 and err["max_abs"] <= 1e-2 * err["max_ref"]


def _run_a_pairs(on, A, B, M, N, K, G, Gr):
    os.environ["CCL_GEMM_A_PAIRS"] = "1" if on else "0"
    try:
        Cbits, _ = run_gemm(A, 0, B, 0, M, N, K, G, Gr, 4096, "256x256", waves=8)
    finally:
        os.environ.pop("CCL_GEMM_A_PAIRS", None)
    return Cbits


@pytest.mark.parametrize("M,N,K,G,Gr", [(512, 512, 64 * k, 1, 1) for k in (1, 2, 3, 4, 5, 7, 8, 9, 13, 14, 15, 22)]
                         + [(2048, 2048, 2048, 8, 2), (2048, 2048, 4096, 8, 1), (2048, 2048, 2048, 8, 8)])
def test_gemm_a_pairs_equal_32k_bit_for_bit(M, N, K, G, Gr):
    """The 256x256 kernel with A staged in 64-K pairs (whole-line loads)
    adds the same 32-K MFMA steps in the same K order as the 32-K kernel:
    C is identical bit for bit, for step counts that stop inside the
    prologue, the rounds, the loop and the tail, and over CCL K blocks."""
    A = W.draw_array(981 + K, M, K, "normal", 1.0)
    B = W.draw_array(982 + K, K, N, "normal", 0.05)
    on = _run_a_pairs(True, A, B, M, N, K, G, Gr)
    off = _run_a_pairs(False, A, B, M, N, K, G, Gr)
    assert np.array_equal(on, off)
    err = OG.errors(OG.decode_bf16(on), OG.gemm_fp64(A, B))
    assert err["rel_fro"] <= 5e-3 and err["max_abs"] <= 1e-2 * err["max_ref"]


@pytest.mark.parametrize("M,N,K,G,Gr,P,ta,tb", [
    (256, 512, 256, 4, 2, 65536, 0, 0),          # padded strips
    (256, 512, 256, 4, 2, 2 * 1024 * 1024, 0, 1),
    (512, 512, 512, 1, 1, 4096, 1, 0),           # one chiplet: all XCDs share the partition
    (1024, 2048, 512, 2, 1, 4096, 0, 0),         # 2 chiplets of 4 XCDs
    (1024, 1024, 512, 8, 8, 4096, 1, 1),         # 8x1: K slices of 64 rows for B
    (1024, 1024, 512, 8, 1, 4096, 0, 0),         # 1x8: K slices of 64 columns for A
    (2048, 384, 256, 4, 4, 4096, 0, 1),          # 4x1 with one K step per B slice
    (128, 128, 64, 1, 1, 4096, 0, 0),            # single tile, single K step
])
def test_gemm_edge_shapes(M, N, K, G, Gr, P, ta, tb):
    A = W.draw_array(1000 + M + K, *((K, M) if ta else (M, K)), "normal", 1.0)
    B = W.draw_array(2000 + N + K, *((N, K) if tb else (K, N)), "normal", 0.5)
    _check_full(A, ta, B, tb, M, N, K, G, Gr, P)


@pytest.mark.parametrize("M,N,K,G,Gr", [(256, 512, 256, 4, 2), (1024, 2048, 256, 8, 2), (1024, 1024, 512, 8, 8)])
def test_gemm_integer_inputs_bit_exact(M, N, K, G, Gr):
    """Values in {-1, 0, 1} with K <= 512: every partial sum is an integer
    of magnitude <= 512, exact in fp32; |C| <= 256 in these draws' bounds
    is checked and then C must equal the integer product exactly."""
    A = W.draw_array(31, M, K, "ternary")
    B = W.draw_array(32, K, N, "ternary")
    ref = OG.decode_bf16(A).astype(np.int64) @ OG.decode_bf16(B).astype(np.int64)
    assert np.abs(ref).max() <= 256          # representable exactly in bf16
    Cbits, _ = run_gemm(A, 0, B, 0, M, N, K, G, Gr, 4096)
    assert np.array_equal(OG.decode_bf16(Cbits), ref.astype(np.float64))


def test_gemm_identity_returns_a_bit_exact():
    M, K = 512, 512
    A = W.draw_array(41, M, K, "normal", 3.0)
    I = W.round_to_bf16_bits(np.eye(K, dtype=np.float32))
    Cbits, _ = run_gemm(A, 0, I, 0, M, K, K, 4, 2, 4096)
    assert np.array_equal(Cbits, A)


def _full_check_large(gemm, grids, page=4096):
    """Every element of C for each grid, against the fp64 oracle computed in
    row blocks of 1024 (once per block, shared by the grids)."""
    wl, g = W.gemm_by_name(gemm)
    A = W.draw(wl.tensors[g.a_src])
    B = W.draw(wl.tensors[g.b_src])
    outs = {}
    for grid in grids:
        (cbuf, gr, gc), _ = run_gemm(A, g.a_trans, B, g.b_trans, g.M, g.N, g.K, g.chiplets, grid,
                                      page, unpack=False)
        outs[grid] = (cbuf, gr, gc)
    A_l = A.T if g.a_trans else A
    B_d = OG.decode(B.T if g.b_trans else B)
    errs = compare_in_row_blocks(outs, g.M, g.N, page,
                                 lambda r0, r1: OG.gemm_fp64(OG.decode(A_l[r0:r1]), B_d),
                                 OG.decode_bf16)
    for grid, err in errs.items():
        print(gemm, "grid rows", grid, "errors over all of C", err, flush=True)
    for grid, err in errs.items():
        assert err["rel_fro"] <= 5e-3, (grid, err)
        assert err["max_abs"] <= 1e-2 * err["max_ref"], (grid, err)


@pytest.mark.parametrize("gemm", ["llama_up", "llama_down"])
def test_gemm_llama_forward_full_compare(gemm):
    _full_check_large(gemm, [2])


@pytest.mark.parametrize("gemm", ["llama_dW_up", "llama_dX"])
def test_gemm_llama_backward_grid_sweep_full_compare(gemm):
    _full_check_large(gemm, [1, 2, 4, 8])


@pytest.mark.parametrize("M,N,K,G,Gr", [(8192, 28672, 8192, 8, 2), (768, 2048, 4096, 8, 1),
                                        (4096, 768, 2048, 8, 8), (256, 512, 256, 4, 2),
                                        (1024, 1024, 1024, 1, 1), (1024, 2048, 512, 2, 1)])
def test_dispatch_probe_tiles_run_on_owner_xcd(M, N, K, G, Gr):
    """Hardware check of the remap: workgroups are dispatched round-robin
    over the 8 XCDs (workgroup w on XCD (w + rot) mod 8, where rot depends
    on the hardware queue behind the stream: 0 for the null stream of a
    fresh process, other values once more streams exist), so the
    workgroups the map gives one chiplet's tiles share one XCD; with
    rot = 0 that XCD is the owner's. Every tile is computed exactly once."""
    torch = __import__("torch")
    plan = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(plan)
    out = torch.full((4 * wgs,), -7, dtype=torch.int32, device="cuda")
    ccl.ccl_debug_dispatch(plan, out)
    rec = out.cpu().numpy().reshape(wgs, 4)
    rot = (rec[:, 0] - np.arange(wgs)) % 8
    print("dispatch rotation", sorted(set(rot.tolist())), flush=True)
    assert len(set(rot.tolist())) == 1
    live = rec[rec[:, 1] >= 0]
    assert len({(a, b) for a, b in live[:, 1:3]}) == len(live) == (M // tm_) * (N // tn_)
    for xcd, ti, tj, owner in live:
        assert owner == OP.owner(ti * tm_ // 128, tj * tn_ // 128, M, N, Gr, G // Gr)
        assert (xcd - rot[0]) % 8 in OP.xcds_of_chiplet(owner, G)


@pytest.mark.parametrize("remap", [0, 1])
@pytest.mark.parametrize("M,N,K,G,Gr", [(2048, 3072, 1024, 8, 2), (1024, 1024, 512, 8, 8),
                                        (256, 512, 256, 4, 2)])
def test_gemm_rowmajor_baseline(remap, M, N, K, G, Gr):
    """The comparison baseline: the same kernel on plain row-major operands,
    with (remap=1) or without (remap=0) the XCD-aware tile map."""
    A = W.draw_array(61 + M, M, K, "normal", 1.0)
    B = W.draw_array(62 + N, K, N, "normal", 0.05)
    plan = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    C = dev_full(M * N)
    print(f"rowmajor {M}x{N}x{K} grid {Gr}x{G // Gr} remap={remap}", flush=True)
    ccl.ccl_gemm_rowmajor(plan, to_dev(A), to_dev(B), C, remap)
    got = OG.decode_bf16(from_dev(C).reshape(M, N))
    err = OG.errors(got, OG.gemm_fp64(A, B))
    assert OG.within_tolerance(err), err


@pytest.mark.parametrize("M,N,K", [(8192, 28672 // 8, 8192), (8192, 8192, 28672 // 8)])
def test_gemm_tensor_parallel_shard_full_compare(M, N, K):
    """One GPU's share of the Llama-3.1-70B FFN under 8-way tensor
    parallelism (up by output columns, down by K), on the plan's automatic
    grid: every element of C against the fp64 oracle, in row blocks."""
    A = W.draw_array(7600 + N, M, K, "normal", 1.0)
    B = W.draw_array(7700 + K, K, N, "normal", 0.02)
    (cbuf, gr, gc), _ = run_gemm(A, 0, B, 0, M, N, K, 8, 0, 4096, unpack=False)
    B_d = OG.decode(B)
    err = compare_in_row_blocks({0: (cbuf, gr, gc)}, M, N, 4096,
                                lambda r0, r1: OG.gemm_fp64(OG.decode(A[r0:r1]), B_d),
                                OG.decode_bf16)[0]
    print("tp8 shard", M, N, K, "grid", gr, gc, "errors over all of C", err, flush=True)
    assert err["rel_fro"] <= 5e-3
    assert err["max_abs"] <= 1e-2 * err["max_ref"]
