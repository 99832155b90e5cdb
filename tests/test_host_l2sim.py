"""CPU tests of the library's finite-L2 traffic model (ccl_remote_bytes_l2)
against the oracle (oracle/l2sim.py), bit for bit.

  * small shapes: every placement, stored-transpose mask, capacity,
    traversal, wave size and K step, against the oracle run live (ragged K
    steps, CCL blocks that are not line-aligned, odd grids, page sizes);
  * the Qwen3 workload GEMMs under three L2 settings: against records the
    oracle wrote (tests/golden/l2_golden.json, make_l2_golden.py);
  * the Llama-3.1-70B forward GEMM at full size: properties that hold at any
    size (capacity 0 is the tile-charge model, which is itself bit-exact to
    the oracle; CCL writes C locally; per-chiplet sums; misses <= accesses).
"""
import json
import os

import pytest

from oracle import l2sim as L
from paper_2606_11718_amd import ccl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden", "l2_golden.json")
PLACE = {"rr": ccl.CCL_PLACE_RR, "coarse": ccl.CCL_PLACE_COARSE, "ccl": ccl.CCL_PLACE_CCL}
TRAV = {"row": 0, "col": 1, "group": 2}


def _both(M, N, K, G, Gr, P, placement, ta, tb, c_read=False, **cfg):
    plan = ccl.ccl_plan(M, N, K, G, Gr, P)
    flags = ta | (tb << 1) | (ccl.CCL_TRAFFIC_C_READ if c_read else 0)
    lib = ccl.ccl_remote_bytes_l2(plan, PLACE[placement], flags,
                                  l2_bytes=cfg["l2_bytes"], slots=cfg["slots"], ways=cfg["ways"],
                                  line_bytes=cfg.get("line", 128), k_step=cfg["k_step"],
                                  traversal=TRAV[cfg["traversal"]],
                                  group_rows=cfg.get("group_rows", 0))
    ora = L.simulate(M, N, K, Gr, G // Gr, P, placement, ta, tb, l2_bytes=cfg["l2_bytes"],
                     slots=cfg["slots"], ways=cfg["ways"], line=cfg.get("line", 128),
                     k_step=cfg["k_step"], traversal=cfg["traversal"], c_read=c_read,
                     group_rows=cfg.get("group_rows", 0))
    return lib, ora


SMALL = [
    # M, N, K, G, Gr, P
    (256, 512, 256, 4, 2, 4096),      # the tiny workload
    (512, 256, 192, 2, 2, 4096),      # K = 3 steps of 64, 1 step of 128 + ragged 64
    (256, 512, 192, 4, 1, 4096),      # CCL blocks of A are 48 elements: not line-aligned
    (384, 768, 384, 3, 1, 2048),      # G = 3
    (256, 256, 320, 2, 1, 65536),     # large pages
    (256, 256, 128, 1, 1, 128),       # one chiplet, page = line
]
CFGS = [
    dict(l2_bytes=0, ways=16, slots=1, k_step=64, traversal="row"),
    dict(l2_bytes=4 * 16 * 128, ways=16, slots=2, k_step=64, traversal="row"),
    dict(l2_bytes=8 * 4 * 128, ways=4, slots=3, k_step=128, traversal="col"),
    dict(l2_bytes=64 * 8 * 128, ways=8, slots=4, k_step=32, traversal="row"),
    dict(l2_bytes=1 * 256 * 128, ways=256, slots=2, k_step=64, traversal="col"),   # fully associative
    dict(l2_bytes=8 * 8 * 128, ways=8, slots=3, k_step=64, traversal="group", group_rows=1),
    dict(l2_bytes=16 * 4 * 128, ways=4, slots=2, k_step=128, traversal="group", group_rows=3),
]


@pytest.mark.parametrize("shape", SMALL)
@pytest.mark.parametrize("placement", ["rr", "coarse", "ccl"])
def test_small_shapes_match_oracle(shape, placement):
    M, N, K, G, Gr, P = shape
    for mask in range(4):
        for cfg in CFGS:
            lib, ora = _both(M, N, K, G, Gr, P, placement, mask & 1, mask >> 1, **cfg)
            assert lib == ora, (shape, placement, mask, cfg)


@pytest.mark.parametrize("placement", ["rr", "coarse", "ccl"])
def test_c_read_matches_oracle(placement):
    for cfg in CFGS[:3]:
        lib, ora = _both(256, 512, 256, 4, 2, 4096, placement, 0, 1, c_read=True, **cfg)
        assert lib == ora


def test_line_sizes_match_oracle():
    for line in (64, 256):
        cfg = dict(l2_bytes=16 * 4 * line, ways=4, slots=2, k_step=64, traversal="row", line=line)
        for placement in ("rr", "ccl"):
            lib, ora = _both(256, 512, 256, 4, 2, 4096, placement, 1, 0, **cfg)
            assert lib == ora


def _golden():
    if not os.path.exists(GOLDEN):
        pytest.skip("l2_golden.json not generated")
    return json.load(open(GOLDEN))["records"]


def test_qwen_workloads_match_oracle_golden():
    recs = _golden()
    assert len(recs) >= 50
    for r in recs:
        plan = ccl.ccl_plan(r["M"], r["N"], r["K"], r["chiplets"], r["grid_rows"], r["page"])
        got = ccl.ccl_remote_bytes_l2(plan, PLACE[r["placement"]], r["trans_a"] | (r["trans_b"] << 1),
                                      l2_bytes=r["l2_bytes"], slots=r["slots"], ways=r["ways"],
                                      line_bytes=r["line"], k_step=r["k_step"],
                                      traversal=TRAV[r["traversal"]])
        for k in ("accesses", "misses", "remote", "remote_per_chiplet"):
            assert got[k] == r[k], (r["gemm"], r["chiplets"], r["l2_bytes"], r["placement"],
                                    r["traversal"], k)


def test_llama_full_size_properties():
    plan = ccl.ccl_plan(8192, 28672, 8192, 8, 2, 4096)
    accessed = None
    for name, pl in PLACE.items():
        charge = ccl.ccl_remote_bytes(plan, pl, 0)
        none = ccl.ccl_remote_bytes_l2(plan, pl, 0, l2_bytes=0, slots=32)
        assert none["remote"] == charge["remote"], name
        assert none["remote_per_chiplet"] == charge["remote_per_chiplet"], name
        assert [a * 128 for a in none["accesses"]] == charge["accessed"][:2]
        accessed = none["accesses"]
    rec = ccl.ccl_remote_bytes_l2(plan, ccl.CCL_PLACE_CCL, 0, l2_bytes=4 << 20, slots=32)
    assert rec["accesses"] == accessed
    assert all(m <= a for m, a in zip(rec["misses"], rec["accesses"]))
    assert rec["remote"][2] == 0
    assert sum(rec["remote_per_chiplet"]) == sum(rec["remote"])
    floor = ccl.ccl_remote_bytes(plan, ccl.CCL_PLACE_CCL, 0)["floor"]
    assert 0 < sum(rec["remote"]) <= floor


@pytest.mark.parametrize("M,N,K,group_rows", [(8192, 28672, 8192, 16), (8192, 8192, 28672, 8)])
def test_kernel_schedule_misses_reach_the_panel_floor(M, N, K, group_rows):
    """The GEMM kernel's own schedule on MI355X, in model terms: 32 resident
    256x256 tiles per XCD = 128 model tiles, a grouped raster of 8 (up) or 4
    (down) kernel tile rows, K steps of 32, a 4 MB 16-way L2 of 128-byte
    lines. With CCL operands every wave of 32 kernel tiles touches 12 panels
    of 256 x K bf16 once: misses = 8 XCDs x waves x 12 x 256 K 2 bytes, the
    fetch the hardware counters measure for these launches (5.64 GB)."""
    plan = ccl.ccl_plan(M, N, K, 8, 2, 4096)
    r = ccl.ccl_remote_bytes_l2(plan, ccl.CCL_PLACE_CCL, 0, l2_bytes=4 << 20, slots=128, ways=16,
                                line_bytes=128, k_step=32, traversal=2, group_rows=group_rows)
    waves = (M // 2 // 256) * (N // 4 // 256) // 32
    assert (r["misses"][0] + r["misses"][1]) * 128 == 8 * waves * 12 * 256 * K * 2


@pytest.mark.parametrize("bad", [
    dict(l2_bytes=3 * 16 * 128),          # 3 sets
    dict(l2_bytes=1000),                  # not whole sets
    dict(l2_bytes=-1),
    dict(ways=0),
    dict(line_bytes=96),                  # not a power of two
    dict(line_bytes=8192),                # larger than the 4 KB page
    dict(slots=0),
    dict(k_step=0),
    dict(traversal=3),
    dict(traversal=2),                    # grouped raster without a group height
    dict(traversal=2, group_rows=-1),
    dict(threads=-1),
    dict(l2_bytes=(1 << 25) * 128, ways=1),   # more than 2^24 lines
])
def test_rejects_bad_config(bad):
    plan = ccl.ccl_plan(256, 512, 256, 4, 2, 4096)
    kw = dict(l2_bytes=1 << 20, slots=4)
    kw.update(bad)
    with pytest.raises(ccl.CCLError) as ei:
        ccl.ccl_remote_bytes_l2(plan, ccl.CCL_PLACE_RR, 0, **kw)
    assert ei.value.status == 1


def test_rejects_bad_placement_and_mask():
    plan = ccl.ccl_plan(256, 512, 256, 4, 2, 4096)
    for pl, mask in ((3, 0), (-1, 0), (0, 8), (0, -1)):
        with pytest.raises(ccl.CCLError) as ei:
            ccl.ccl_remote_bytes_l2(plan, pl, mask, l2_bytes=0, slots=1)
        assert ei.value.status == 1


def test_thread_count_does_not_change_result():
    plan = ccl.ccl_plan(1024, 2048, 512, 8, 2, 4096)
    one = ccl.ccl_remote_bytes_l2(plan, ccl.CCL_PLACE_RR, 0, l2_bytes=64 << 10, slots=8, threads=1)
    many = ccl.ccl_remote_bytes_l2(plan, ccl.CCL_PLACE_RR, 0, l2_bytes=64 << 10, slots=8, threads=8)
    assert one == many
