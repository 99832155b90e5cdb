"""GPU checks of ccl_debug_gemm_timeline: the profiling launch computes the
same C as ccl_gemm, bit for bit, and every wave's record is well formed.

The record layout (per wave, 8 uint64): real-time counter at start, after
the prologue, after the K loop and after the stores' issue; shader clock at start
and after the K loop; XCD id; raw HW_ID. The owner check is the Sec. III-A
co-location that the dispatch probe also checks.
"""
import numpy as np
import pytest

import workloads as W
from oracle import plan as OP
from paper_2606_11718_amd import ccl
from tests.helpers import dev_full, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,N,K,G,Gr", [(768, 2048, 4096, 8, 1), (4096, 768, 2048, 8, 8),
                                        (2048, 2048, 1024, 8, 2), (256, 512, 256, 4, 2)])
def test_timeline_matches_gemm_and_is_well_formed(M, N, K, G, Gr):
    torch = __import__("torch")
    plan = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    tm_, tn_, wgs = ccl.ccl_debug_gemm_config(plan)
    print(f"timeline {M}x{N}x{K} G={G} Gr={Gr} tile {tm_}x{tn_} wgs={wgs}", flush=True)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    A = to_dev(W.draw_array(71, 1, la.total_bytes // 2, "normal", 1.0)[0])
    B = to_dev(W.draw_array(72, 1, lb.total_bytes // 2, "normal", 0.05)[0])
    C1, C2 = dev_full(lc.total_bytes // 2), dev_full(lc.total_bytes // 2)
    waves = 8
    tl = torch.zeros(wgs * waves * 8, dtype=torch.int64, device="cuda")
    ccl.ccl_gemm(plan, A, B, C1)
    ccl.ccl_debug_gemm_timeline(plan, A, B, C2, tl, tl.numel() * 8)
    assert np.array_equal(from_dev(C1), from_dev(C2))
    rec = tl.cpu().numpy().reshape(wgs, waves, 8)
    live = [w for w in range(wgs) if ccl.ccl_debug_tile_of_wg(plan, w)[1] >= 0]
    dead = [w for w in range(wgs) if w not in set(live)]
    assert np.all(rec[dead] == 0)
    r = rec[live]
    assert np.all(r[:, :, 0] > 0)
    assert np.all(np.diff(r[:, :, 0:4], axis=2) >= 0)           # phases in order
    assert np.all(r[:, :, 5] > r[:, :, 4])                       # clock advanced over the loop
    assert np.all(r[:, :, 6] == r[:, :1, 6])                     # one XCD and one CU per workgroup
    assert np.all(r[:, :, 7] & 0xFF00 == r[:, :1, 7] & 0xFF00)
    # Round-robin dispatch: workgroup w on XCD (w + rot) mod 8, one rotation
    # for the launch, set by the hardware queue behind the stream.
    xcc = r[:, 0, 6] & 0xF
    rot = (xcc - np.array(live)) % 8
    print("dispatch rotation", sorted(set(rot.tolist())), flush=True)
    assert len(set(rot.tolist())) == 1
    for w, row in zip(live, r):
        xcd, ti, tj = ccl.ccl_debug_tile_of_wg(plan, w)
        assert xcd == w % 8 and (row[0, 6] & 0xF) == (xcd + rot[0]) % 8
        owner = OP.owner(ti * tm_ // 128, tj * tn_ // 128, M, N, Gr, G // Gr)
        assert xcd in OP.xcds_of_chiplet(owner, G)
    # the clock implied by the loop (shader cycles over 100 MHz ticks) is a
    # plausible GPU clock
    dt = (r[:, :, 2] - r[:, :, 1]).astype(np.float64)
    ok = dt > 100
    if ok.any():
        ghz = (r[:, :, 5] - r[:, :, 4])[ok] / ((r[:, :, 2] - r[:, :, 0])[ok] * 10.0)
        assert 0.3 < np.median(ghz) < 3.0, np.median(ghz)


def test_timeline_refuses_short_buffer_and_fp8():
    torch = __import__("torch")
    plan = ccl.ccl_plan(256, 512, 256, 4, 2, 4096)
    _, _, wgs = ccl.ccl_debug_gemm_config(plan)
    la, lb, lc = (ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C))
    A, B, C = (dev_full(x.total_bytes // 2) for x in (la, lb, lc))
    tl = torch.zeros(wgs * 8 * 8, dtype=torch.int64, device="cuda")
    with pytest.raises(RuntimeError, match="timeline smaller"):
        ccl.ccl_debug_gemm_timeline(plan, A, B, C, tl, tl.numel() * 8 - 8)
    f8 = ccl.ccl_plan_typed(256, 512, 256, 4, 2, 4096, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_BF16)
    with pytest.raises(RuntimeError, match="bf16"):
        ccl.ccl_debug_gemm_timeline(f8, A, B, C, tl, tl.numel() * 8)
    torch.cuda.synchronize()
