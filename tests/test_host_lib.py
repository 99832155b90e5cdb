"""CPU tests of the HIP library's host side, through the C ABI.

No GPU: the library loads, exports every symbol the header declares, and its
host-only calls (plan, layouts, remote-byte model, workgroup -> tile map)
match the oracle bit for bit.
"""
import ctypes
import json
import os
import re

import numpy as np
import pytest

from oracle import layout as OL
from oracle import plan as OP
from oracle import traffic as OT
from paper_2606_11718_amd import ccl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ccl.h")
GOLDEN = os.path.join(ROOT, "tests", "golden", "traffic_golden.json")
PLACE = {"rr": ccl.CCL_PLACE_RR, "coarse": ccl.CCL_PLACE_COARSE, "ccl": ccl.CCL_PLACE_CCL}


def header_functions():
    text = open(HEADER).read()
    return re.findall(r"^(?:ccl_status|const char\*)\s+(ccl_\w+)\(", text, re.M)


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 10
    ccl.library()          # loads the HIP runtime torch uses, then libccl.so
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_11718_amd", "libccl.so"))
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(ccl.EXPORTED)


def test_status_strings():
    assert ccl.ccl_status_string(0) == "CCL_OK"
    assert ccl.ccl_status_string(2) == "CCL_ERR_UNALIGNED_PARTITION"
    assert ccl.ccl_status_string(99) == "CCL_ERR_UNKNOWN"


@pytest.mark.parametrize("args,status", [
    ((0, 512, 256, 4, 2, 4096), 1),          # empty M
    ((256, 512, 0, 4, 2, 4096), 1),          # empty K
    ((256, 512, 256, 0, 0, 4096), 1),        # no chiplets
    ((256, 512, 256, 65, 0, 4096), 1),       # too many chiplets
    ((256, 512, 256, 4, 3, 4096), 1),        # grid does not divide
    ((256, 512, 256, 4, -1, 4096), 1),
    ((256, 512, 256, 4, 2, 3000), 1),        # page not a power of two
    ((256, 512, 256, 4, 2, 64), 1),          # page too small
    ((256, 512, 256, 4, 4, 4096), 2),        # 256 rows / 4 is not a tile
    ((256, 500, 256, 4, 2, 4096), 2),        # ragged N
    ((256, 512, 255, 4, 2, 4096), 2),        # K not divisible by the grid
    ((100, 100, 100, 8, 0, 4096), 2),        # automatic: no aligned grid
    ((1 << 31, 128, 128, 1, 1, 4096), 1),    # overflow guard
])
def test_plan_rejections(args, status):
    with pytest.raises(ccl.CCLError) as ei:
        ccl.ccl_plan(*args)
    assert ei.value.status == status
    assert ccl.ccl_last_error() != ""


def test_null_arguments_are_rejected_without_gpu():
    p = ccl.ccl_plan(256, 512, 256, 4, 2, 4096)
    lib = ccl.library()
    assert lib.ccl_plan_layout(p, 0, None) == 1
    assert lib.ccl_plan_layout(p, 7, ctypes.byref(ccl._Layout())) == 1
    assert lib.ccl_remote_bytes(p, 5, 0, ctypes.byref(ccl._Traffic())) == 1
    assert lib.ccl_remote_bytes(p, 0, 8, ctypes.byref(ccl._Traffic())) == 1
    assert lib.ccl_remote_bytes(p, 0, -1, ctypes.byref(ccl._Traffic())) == 1
    assert lib.ccl_gemm(p, None, None, None, None) == 1
    assert lib.ccl_gemm(p, 16, 32, 8, None) == 4            # misaligned pointer
    assert lib.ccl_pack(p, 0, None, 256, 0, None, None) == 1
    assert lib.ccl_pack(p, 2, 16, 512, 1, 16, None) == 1     # C has no transpose
    assert lib.ccl_pack(p, 0, 16, 100, 0, 16, None) == 1     # ld < cols
    assert lib.ccl_unpack(p, 1, 16, 16, 10, None) == 1
    assert lib.ccl_gemm_rowmajor(p, 16, 16, 16, 2, None) == 1    # remap must be 0/1
    assert lib.ccl_gemm_rowmajor(p, 16, 32, 8, 1, None) == 4     # misaligned
    assert lib.ccl_plan_destroy(None) == 0
    q = ccl.ccl_plan(256, 512, 208, 4, 2, 4096)             # K / Gc = 104: no GEMM kernel
    with pytest.raises(ccl.CCLError) as ei:
        ccl.ccl_gemm(q, 16, 16, 16)
    assert ei.value.status == 3


LAYOUT_CASES = [(256, 512, 256, 4, 2, 4096), (4096, 1536, 2048, 8, 2, 4096),
                (768, 2048, 4096, 8, 1, 65536), (384, 768, 201, 3, 1, 2048),
                (256, 512, 256, 4, 2, 2 * 1024 * 1024)]


@pytest.mark.parametrize("M,N,K,G,Gr,P", LAYOUT_CASES)
def test_layouts_match_oracle(M, N, K, G, Gr, P):
    p = ccl.ccl_plan(M, N, K, G, Gr, P)
    Gc = G // Gr
    for op, name in ((ccl.CCL_A, "A"), (ccl.CCL_B, "B"), (ccl.CCL_C, "C")):
        R, Cc = OL.operand_shape(name, M, N, K)
        lay = ccl.ccl_plan_layout(p, op)
        hr, wc = OL.block_shape(R, Cc, Gr, Gc)
        assert (lay.rows, lay.cols, lay.grid_r, lay.grid_c) == (R, Cc, Gr, Gc)
        assert (lay.block_rows, lay.block_cols) == (hr, wc)
        assert lay.strip_stride_bytes == OL.strip_stride_bytes(R, Cc, Gr, Gc, P)
        assert lay.total_bytes == OL.total_bytes(R, Cc, Gr, Gc, P)


@pytest.mark.parametrize("M,N,K,G", [(768, 2048, 4096, 8), (4096, 768, 2048, 8), (1024, 4096, 1024, 8),
                                     (4096, 1024, 1024, 8), (256, 512, 256, 4), (8192, 28672, 8192, 8),
                                     (512, 512, 512, 1), (1024, 1024, 1024, 2)])
def test_auto_grid_matches_oracle(M, N, K, G):
    p = ccl.ccl_plan(M, N, K, G, 0, 4096)
    assert ccl.ccl_plan_grid(p)[0] == OP.auto_grid_rows(M, N, K, G)


def _golden_records():
    if not os.path.exists(GOLDEN):
        pytest.skip("traffic_golden.json not generated")
    return json.load(open(GOLDEN))["records"]


def test_remote_bytes_match_oracle_golden_all_workloads():
    """Every workload GEMM x grid x page x placement, bit-exact."""
    recs = _golden_records()
    assert len(recs) >= 90
    for r in recs:
        p = ccl.ccl_plan(r["M"], r["N"], r["K"], r["chiplets"], r["grid_rows_requested"], r["page"])
        assert ccl.ccl_plan_grid(p)[0] == r["grid_rows"]
        got = ccl.ccl_remote_bytes(p, PLACE[r["placement"]], r["trans_a"] | (r["trans_b"] << 1))
        for k in ("accessed", "remote", "remote_per_chiplet", "floor", "footprint"):
            assert got[k] == r[k], (r["gemm"], r["grid_rows"], r["page"], r["placement"], k)


RANDOM_SHAPES = [
    (256, 512, 256, 2, 2, 4096, 0, 0), (256, 256, 384, 1, 2, 256, 1, 0), (512, 256, 192, 4, 1, 512, 1, 1),
    (384, 768, 201, 1, 3, 2048, 1, 0), (1024, 256, 320, 8, 1, 128, 0, 1), (256, 1024, 96, 1, 8, 65536, 0, 0),
    (640, 384, 330, 5, 1, 1024, 1, 1), (256, 384, 300, 2, 3, 128, 0, 1), (128, 128, 7, 1, 1, 128, 1, 1),
]


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", RANDOM_SHAPES)
@pytest.mark.parametrize("placement", OT.PLACEMENTS)
def test_remote_bytes_match_oracle_small(M, N, K, Gr, Gc, P, ta, tb, placement):
    p = ccl.ccl_plan(M, N, K, Gr * Gc, Gr, P)
    for c_read in (False, True):
        flags = ta | (tb << 1) | (ccl.CCL_TRAFFIC_C_READ if c_read else 0)
        got = ccl.ccl_remote_bytes(p, PLACE[placement], flags)
        ref = OT.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb, c_read=c_read)
        for k in ("accessed", "remote", "remote_per_chiplet", "floor", "footprint"):
            assert got[k] == ref[k], (k, c_read)


TILE_CASES = [(256, 512, 256, 4, 2), (4096, 1536, 2048, 8, 2), (768, 2048, 4096, 8, 1),
              (4096, 768, 2048, 8, 8), (8192, 28672, 8192, 8, 2), (8192, 8192, 28672, 8, 4),
              (1024, 1024, 1024, 1, 1), (1024, 2048, 512, 2, 1), (2048, 384, 256, 4, 4)]


@pytest.mark.parametrize("M,N,K,G,Gr", TILE_CASES)
def test_workgroup_tile_map_covers_each_tile_once_on_owner_xcd(M, N, K, G, Gr):
    """Round-robin dispatch puts workgroup w on XCD w mod 8; the map must send
    every kernel tile exactly once to an XCD of the chiplet owning it."""
    p = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    Gc = G // Gr
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(p)
    assert wgs % 8 == 0
    seen = {}
    for wg in range(wgs):
        xcd, ti, tj = ccl.ccl_debug_tile_of_wg(p, wg)
        assert xcd == wg % 8
        if ti < 0:
            continue
        assert (ti, tj) not in seen
        seen[(ti, tj)] = xcd
        owner = OP.owner(ti * tm_ // 128, tj * tn_ // 128, M, N, Gr, Gc)
        # every 128x128 model tile inside the kernel tile has the same owner
        assert owner == OP.owner((ti * tm_ + tm_ - 1) // 128, (tj * tn_ + tn_ - 1) // 128, M, N, Gr, Gc)
        assert xcd in OP.xcds_of_chiplet(owner, G)
    assert len(seen) == (M // tm_) * (N // tn_)
    # workgroups beyond the launch have no tile
    assert ccl.ccl_debug_tile_of_wg(p, wgs)[1] == -1


@pytest.mark.parametrize("M,N,K,G,Gr", [(8192, 28672, 8192, 8, 2), (8192, 8192, 28672, 8, 2),
                                        (8192, 28672, 8192, 8, 1), (8192, 8192, 28672, 8, 1)])
def test_resident_tiles_share_twelve_panels(M, N, K, G, Gr):
    """Each XCD runs 32 of its 256x256 tiles at once (one workgroup per CU,
    in slot order). Where the partition's tile columns allow it (a multiple
    of 8, or of 4 with a multiple of 8 tile rows), every such wave must cover
    a 4x8 or 8x4 block of tiles: 12 distinct A row panels plus B column
    panels, never a wave split over two raster groups. Otherwise (14 tile
    columns for dW_up on 1x8) some waves straddle two groups; there the
    plan's height is the one with the fewest panels in total
    (test_raster_height_touches_fewest_panels)."""
    p = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(p)
    assert (tm_, tn_) == (256, 256)
    tiles_m, tiles_n = M // Gr // 256, N // (G // Gr) // 256
    exact = tiles_n % 8 == 0 or (tiles_n % 4 == 0 and tiles_m % 8 == 0)
    slots = wgs // 8
    for xcd in range(8):
        tiles = [ccl.ccl_debug_tile_of_wg(p, xcd + 8 * s)[1:] for s in range(slots)]
        for w in range(0, slots, 32):
            wave = [t for t in tiles[w:w + 32] if t[0] >= 0]
            rows = {t[0] for t in wave}
            cols = {t[1] for t in wave}
            if exact and len(wave) == 32:
                assert len(rows) + len(cols) == 12, (xcd, w, sorted(rows), sorted(cols))
            elif exact:
                assert len(rows) + len(cols) <= 12


def _wave_panels(p):
    """Distinct tile rows plus tile columns of every wave of 32 consecutive
    slots on each XCD, summed (from the plan's workgroup -> tile map)."""
    _, _, wgs = ccl.ccl_debug_gemm_config(p)
    slots, total = wgs // 8, 0
    for xcd in range(8):
        tiles = [ccl.ccl_debug_tile_of_wg(p, xcd + 8 * s)[1:] for s in range(slots)]
        for w in range(0, slots, 32):
            wave = [t for t in tiles[w:w + 32] if t[0] >= 0]
            total += len({t[0] for t in wave}) + len({t[1] for t in wave})
    return total


@pytest.mark.parametrize("M,N,K,G,Gr", [(8192, 28672, 8192, 8, 2), (8192, 8192, 28672, 8, 2),
                                        (8192, 28672, 8192, 8, 1), (8192, 8192, 28672, 8, 1),
                                        (4096, 1536, 2048, 8, 2), (2048, 4096, 1024, 4, 2)])
def test_raster_height_touches_fewest_panels(M, N, K, G, Gr, monkeypatch):
    """The plan's raster is at least as good as 4- and 8-row groups in
    panels touched per wave, and it is 4 rows on a tie."""
    chosen = _wave_panels(ccl.ccl_plan(M, N, K, G, Gr, 4096))
    forced = {}
    for gm in (4, 8):
        monkeypatch.setenv("CCL_GEMM_GROUP_M", str(gm))
        forced[gm] = _wave_panels(ccl.ccl_plan(M, N, K, G, Gr, 4096))
    monkeypatch.delenv("CCL_GEMM_GROUP_M")
    assert chosen == min(forced.values())
    if forced[4] == forced[8]:
        assert chosen == forced[4]


def test_gemm_config_tiles_nest_in_partitions():
    for (M, N, K, G, Gr) in TILE_CASES:
        p = ccl.ccl_plan(M, N, K, G, Gr, 4096)
        tm_, tn_, _ = ccl.ccl_debug_gemm_config(p)
        assert (M // Gr) % tm_ == 0 and (N // (G // Gr)) % tn_ == 0
        assert tm_ in (128, 256) and tn_ in (128, 256)


@pytest.mark.parametrize("T,D,F,G,Gr", [(8192, 8192, 28672, 8, 2), (4096, 2048, 1536, 8, 2),
                                        (2048, 1024, 3072, 8, 4), (256, 256, 512, 4, 2)])
def test_ffn_intermediate_needs_no_repack(T, D, F, G, Gr):
    """C of X[T x D] W1[D x F] and A of H[T x F] W2[F x D] on the same grid are
    the same CCL layout, so the first GEMM's output buffer is the second
    GEMM's A buffer as it stands (activations produced directly in CCL)."""
    up = ccl.ccl_plan(T, F, D, G, Gr, 4096)
    down = ccl.ccl_plan(T, D, F, G, Gr, 4096)
    assert ccl.ccl_plan_layout(up, ccl.CCL_C) == ccl.ccl_plan_layout(down, ccl.CCL_A)


# ---- element types (fp8 E4M3 / bf16 operands, bf16 / fp32 output) ----------

DT = {1: ccl.CCL_DT_FP8_E4M3, 2: ccl.CCL_DT_BF16, 4: ccl.CCL_DT_FP32}
TYPED = [(1, 2), (1, 4), (2, 4), (2, 2), (4, 4)]  # (e_ab, e_c)


@pytest.mark.parametrize("eab,ec", TYPED)
@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", RANDOM_SHAPES[:6])
def test_typed_layouts_and_remote_bytes_match_oracle(eab, ec, M, N, K, Gr, Gc, P, ta, tb):
    p = ccl.ccl_plan_typed(M, N, K, Gr * Gc, Gr, P, DT[eab], DT[ec])
    for op, e in ((ccl.CCL_A, eab), (ccl.CCL_B, eab), (ccl.CCL_C, ec)):
        lay = ccl.ccl_plan_layout(p, op)
        R, Cc = OL.operand_shape("ABC"[op], M, N, K)
        assert lay.elem_bytes == e
        assert lay.strip_stride_bytes == OL.strip_stride_bytes(R, Cc, Gr, Gc, P, e)
        assert lay.total_bytes == OL.total_bytes(R, Cc, Gr, Gc, P, e)
    for name, pl in PLACE.items():
        got = ccl.ccl_remote_bytes(p, pl, ta | (tb << 1))
        ref = OT.remote_bytes(M, N, K, Gr, Gc, P, name, ta, tb, e=(eab, eab, ec))
        for k in ("accessed", "remote", "remote_per_chiplet", "floor", "footprint"):
            assert got[k] == ref[k], (name, k)


@pytest.mark.parametrize("M,N,K,G", [(768, 2048, 4096, 8), (4096, 768, 2048, 8), (8192, 28672, 8192, 8)])
def test_typed_auto_grid_matches_oracle(M, N, K, G):
    for eab, ec in TYPED:
        p = ccl.ccl_plan_typed(M, N, K, G, 0, 4096, DT[eab], DT[ec])
        assert ccl.ccl_plan_grid(p)[0] == OP.auto_grid_rows(M, N, K, G, e=(eab, eab, ec))


def test_typed_plan_rejects_bad_types():
    for ab, c in ((ccl.CCL_DT_BF16, ccl.CCL_DT_FP8_E4M3), (ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_FP8_E4M3),
                  (3, 0), (0, -1)):
        with pytest.raises(ccl.CCLError) as ei:
            ccl.ccl_plan_typed(256, 512, 256, 4, 2, 4096, ab, c)
        assert ei.value.status == 1


def test_typed_l2_model_matches_oracle():
    from oracle import l2sim as OL2
    for eab, ec, ks in ((1, 2, 128), (1, 4, 128), (2, 4, 64)):
        p = ccl.ccl_plan_typed(256, 512, 512, 4, 2, 4096, DT[eab], DT[ec])
        for name, pl in PLACE.items():
            got = ccl.ccl_remote_bytes_l2(p, pl, 1, l2_bytes=8 * 16 * 128, slots=2, k_step=ks)
            ref = OL2.simulate(256, 512, 512, 2, 2, 4096, name, 1, 0, l2_bytes=8 * 16 * 128, slots=2,
                               k_step=ks, e=(eab, eab, ec))
            assert got == ref, (eab, ec, name)


@pytest.mark.parametrize("M,N,K,G,Gr", [(256, 512, 256, 4, 2), (4096, 1536, 2048, 8, 2), (768, 2048, 4096, 8, 1),
                                        (4096, 768, 2048, 8, 8), (8192, 28672, 8192, 8, 2),
                                        (1024, 768, 1024, 8, 8), (384, 768, 384, 1, 1)])
@pytest.mark.parametrize("c_type", [ccl.CCL_DT_BF16, ccl.CCL_DT_FP32])
def test_gemm_host_checks_pass_for_valid_plans(M, N, K, G, Gr, c_type):
    """Every host-side check of ccl_gemm and ccl_gemm_rowmajor, including the
    one that every element the kernel can address lies inside the operand
    buffers, passes for valid plans of either C type: without a GPU the call
    gets as far as the device query and fails there."""
    import torch
    if torch.cuda.device_count() > 0:      # placeholder pointers must never reach a device
        pytest.skip("needs a host without a GPU")
    lib = ccl.library()
    p = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ccl.CCL_DT_BF16, c_type)
    for st in (lib.ccl_gemm(p, 4096, 4096, 4096, None),
               lib.ccl_gemm_scaled(p, 2.0, 4096, 4096, 1.0, 4096, None),
               lib.ccl_gemm_rowmajor(p, 4096, 4096, 4096, 0, None)):
        msg = lib.ccl_last_error().decode()
        assert "internal" not in msg
        assert st == 5 and "hipGetDevice" in msg, msg


def test_fp32_operand_plan_has_no_gemm():
    p = ccl.ccl_plan_typed(256, 512, 256, 4, 2, 4096, ccl.CCL_DT_FP32, ccl.CCL_DT_FP32)
    assert ccl.ccl_plan_layout(p, ccl.CCL_A).elem_bytes == 4
    lib = ccl.library()
    assert lib.ccl_gemm(p, 4096, 4096, 4096, None) == 3      # unsupported, before any device call
    assert "bf16 or fp8" in lib.ccl_last_error().decode()


def test_size_limits_are_rejected_before_any_launch():
    """Shapes past the kernels' 32-bit in-tile byte offsets, or with a CCL
    strip of 2^31 elements or more, are refused on the host (status
    CCL_ERR_UNSUPPORTED) before any device call."""
    lib = ccl.library()
    wide = ccl.ccl_plan(256, 128, 1 << 23, 1, 1, 4096)      # 255 rows of A span > 2^31 bytes
    assert lib.ccl_gemm(wide, 4096, 4096, 4096, None) == 3
    assert "32-bit" in lib.ccl_last_error().decode()
    assert lib.ccl_gemm_rowmajor(wide, 4096, 4096, 4096, 1, None) == 3
    # B rows of 17.9M bf16: one K step (31 rows) spans 1.1 GB, but four steps
    # of the rounds path (127 rows) span 4.5 GB; the same for fp8's 128-wide step
    for ab, n in ((ccl.CCL_DT_BF16, 128 * 140000), (ccl.CCL_DT_FP8_E4M3, 128 * 140000 * 2)):
        longb = ccl.ccl_plan_typed(128, n, 128, 1, 1, 4096, ab, ccl.CCL_DT_BF16)
        assert lib.ccl_gemm(longb, 4096, 4096, 4096, None) == 3
        assert "32-bit" in lib.ccl_last_error().decode()
        assert lib.ccl_gemm_splitk(longb, 1.0, 4096, 4096, 0.0, 4096, 2, 4096, 1 << 40, None) == 3
        assert "32-bit" in lib.ccl_last_error().decode()
    huge = ccl.ccl_plan(65536, 128, 65536, 1, 1, 4096)      # one strip of 2^32 elements
    assert lib.ccl_pack(huge, ccl.CCL_A, 4096, 65536, 0, 4096, None) == 3
    assert lib.ccl_unpack(huge, ccl.CCL_A, 4096, 4096, 65536, None) == 3


def test_one_plan_from_many_host_threads():
    """A plan is immutable: concurrent host calls on it give the serial results."""
    from concurrent.futures import ThreadPoolExecutor
    p = ccl.ccl_plan(4096, 1536, 2048, 8, 2, 4096)
    want = [ccl.ccl_remote_bytes(p, pl, m) for pl in range(3) for m in range(8)]
    def job(i):
        pl, m = divmod(i % 24, 8)
        return i % 24, ccl.ccl_remote_bytes(p, pl, m)
    with ThreadPoolExecutor(max_workers=8) as ex:
        for i, got in ex.map(job, range(96)):
            assert got == want[i]


@pytest.mark.parametrize("M,N,K,G,Gr,why", [
    (384, 768, 384, 3, 1, "divide the 8"),           # 3 chiplets do not map onto 8 XCDs
    (2048, 1024, 256, 16, 2, "divide the 8"),        # more chiplets than XCDs
    (256, 512, 48, 2, 1, "multiples of 32"),         # K / Gc = 24 is not a whole K step
    (256, 512, 80, 1, 1, "multiples of 32"),         # K = 80: two and a half K steps
])
def test_gemm_unsupported_plans_are_refused_on_the_host(M, N, K, G, Gr, why):
    """Valid plans (layouts and traffic models work) whose GEMM the kernels
    cannot run: ccl_gemm says so before any device call."""
    p = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    assert ccl.ccl_plan_layout(p, ccl.CCL_A).total_bytes > 0
    lib = ccl.library()
    assert lib.ccl_gemm(p, 4096, 4096, 4096, None) == 3
    assert why in lib.ccl_last_error().decode()


def test_fp8_gemm_needs_64_element_k_steps():
    p = ccl.ccl_plan_typed(256, 512, 96, 1, 1, 4096, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_BF16)
    lib = ccl.library()
    assert lib.ccl_gemm(p, 4096, 4096, 4096, None) == 3
    assert "64" in lib.ccl_last_error().decode()
