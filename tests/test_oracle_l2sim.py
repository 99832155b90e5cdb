"""Pins of the oracle's finite-L2 remote-traffic model (Sec. IV-A).

The LRU core is checked against hand-worked sequences and against an
independent rule (a line hits iff fewer than `ways` distinct other lines of
its set were touched since its previous access). The whole model is checked
against two limits it must reduce to:
  * capacity 0 (no cache) is the tile-charge model of oracle.traffic,
    itself pinned by brute force and closed forms;
  * an unbounded cache charges each chiplet once per distinct remote line it
    touches, computed here from element-level chiplet maps.
Plus: misses never grow with associativity (LRU inclusion within a set),
G = 1 gives zero, CCL keeps C writes and the unshared operand local.
"""
import random

import numpy as np
import pytest

from oracle import l2sim as L
from oracle import traffic as T
from oracle import layout
from oracle.plan import TILE, owner


# ---------------------------------------------------------------------------
# set index and LRU core
# ---------------------------------------------------------------------------

def test_fold_set_hand_values():
    assert L.fold_set(0b1011_0110, 16) == 0b0110 ^ 0b1011
    assert L.fold_set(4096 * 3 + 5, 4096) == 5 ^ 3
    assert L.fold_set((7 << 24) | (1 << 12) | 9, 4096) == 9 ^ 1 ^ 7
    assert L.fold_set(123456789, 1) == 0
    assert all(0 <= L.fold_set(x, 64) < 64 for x in range(5000))


def test_lru_hand_sequence_one_set():
    c = L.LRUCache(2 * 128, ways=2, line=128)            # 1 set, 2 ways
    got = [c.access(x) for x in (1, 2, 1, 3, 2, 1)]
    # 1 miss, 2 miss, 1 hit, 3 miss (evicts 2), 2 miss (evicts 1), 1 miss
    assert got == [False, False, True, False, False, False]


def test_lru_hand_sequence_two_sets():
    c = L.LRUCache(2 * 128, ways=1, line=128)            # 2 sets, direct mapped
    # fold with 1 bit: set(0)=0, set(1)=1, set(2)=1, set(3)=0
    got = [c.access(x) for x in (0, 3, 0, 1, 2, 1, 1)]
    assert got == [False, False, False, False, False, False, True]


def test_lru_rejects_bad_geometry():
    with pytest.raises(ValueError):
        L.LRUCache(3 * 128 * 16, ways=16, line=128)      # 3 sets
    with pytest.raises(ValueError):
        L.LRUCache(1000, ways=16, line=128)


def _hits_by_reuse_rule(stream, sets, ways):
    """Independent rule: access i hits iff its line was seen before and fewer
    than `ways` distinct other lines of the same set came in between."""
    out = []
    for i, x in enumerate(stream):
        s = L.fold_set(x, sets)
        prev = max((j for j in range(i) if stream[j] == x), default=None)
        if prev is None:
            out.append(False)
            continue
        between = {y for y in stream[prev + 1:i] if L.fold_set(y, sets) == s}
        out.append(len(between) < ways)
    return out


@pytest.mark.parametrize("sets,ways", [(1, 1), (1, 4), (2, 2), (4, 3), (8, 2)])
def test_lru_matches_reuse_rule(sets, ways):
    rnd = random.Random(1000 * sets + ways)
    for trial in range(6):
        stream = [rnd.randrange(3 * sets * ways + 2) for _ in range(120)]
        c = L.LRUCache(sets * ways * 128, ways=ways, line=128)
        assert [c.access(x) for x in stream] == _hits_by_reuse_rule(stream, sets, ways)


# ---------------------------------------------------------------------------
# the model's limits
# ---------------------------------------------------------------------------

CASES = [
    # M, N, K, Gr, Gc, P, trans_a, trans_b
    (256, 512, 256, 2, 2, 4096, 0, 0),      # tiny workload shape
    (256, 512, 256, 2, 2, 4096, 1, 0),
    (256, 512, 256, 2, 2, 4096, 0, 1),
    (512, 256, 128, 4, 1, 4096, 0, 0),
    (256, 512, 512, 1, 4, 4096, 1, 1),
    (512, 256, 192, 2, 1, 4096, 0, 1),
    (256, 256, 384, 2, 1, 65536, 0, 0),
]
PLACEMENTS = ("rr", "coarse", "ccl")


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("placement", PLACEMENTS)
def test_capacity_zero_is_tile_charge(case, placement):
    M, N, K, Gr, Gc, P, ta, tb = case
    ref = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb)
    for slots, trav, ks in ((1, "row", 64), (3, "col", 128), (2, "group", 64)):   # K step 128: ragged last step
        got = L.simulate(M, N, K, Gr, Gc, P, placement, ta, tb, l2_bytes=0, slots=slots,
                         traversal=trav, k_step=ks, group_rows=1 + (M // 128) // 3)
        assert got["remote"] == ref["remote"]
        assert got["remote_per_chiplet"] == ref["remote_per_chiplet"]
        assert got["misses"] == got["accesses"]
        # every access is a whole 128-byte line of panel data
        assert [a * 128 for a in got["accesses"]] == ref["accessed"][:2]


def test_capacity_zero_charges_whole_lines():
    # CCL blocks of A are 48 elements (96 bytes) wide here, so block rows are
    # not line-aligned: a line counts whole even when half of it is read.
    M, N, K, Gr, Gc, P = 256, 512, 192, 1, 4, 4096
    ref = T.remote_bytes(M, N, K, Gr, Gc, P, "ccl")
    got = L.simulate(M, N, K, Gr, Gc, P, "ccl", l2_bytes=0, slots=1)
    assert got["remote"][0] > ref["remote"][0]
    assert got["accesses"][0] * 128 > ref["accessed"][0]


def _distinct_remote_lines(M, N, K, Gr, Gc, P, placement, ta, tb, e=2):
    """Per chiplet: distinct remote lines over all of its tiles' A and B panels,
    with element homes from the tile-charge model's chip_of."""
    G = Gr * Gc
    total = 0
    trans = {"A": ta, "B": tb}
    for p in range(G):
        lines = {"A": set(), "B": set()}
        for ti in range(M // TILE):
            for tj in range(N // TILE):
                if owner(ti, tj, M, N, Gr, Gc) != p:
                    continue
                for op, rows, cols in (("A", np.arange(ti * TILE, (ti + 1) * TILE), np.arange(K)),
                                       ("B", np.arange(K), np.arange(tj * TILE, (tj + 1) * TILE))):
                    R, Cc = layout.operand_shape(op, M, N, K)
                    r, c = rows[:, None], cols[None, :]
                    if placement == "ccl":
                        off = layout.ccl_offset(r, c, R, Cc, Gr, Gc, P, e)
                    else:
                        off = T.stored_offset(r, c, R, Cc, trans[op], e)
                    chip = T.chip_of(r, c, R, Cc, trans[op], placement, Gr, Gc, P, e)
                    ln = (off // 128)[chip != p]
                    lines[op].update(int(x) for x in np.unique(ln))
        total += 128 * (len(lines["A"]) + len(lines["B"]))
    return total


@pytest.mark.parametrize("case", CASES[:4])
@pytest.mark.parametrize("placement", PLACEMENTS)
def test_unbounded_cache_is_first_touch(case, placement):
    M, N, K, Gr, Gc, P, ta, tb = case
    ways = 1 << 13                       # one fully associative set larger than any panel set
    got = L.simulate(M, N, K, Gr, Gc, P, placement, ta, tb, l2_bytes=ways * 128, ways=ways,
                     slots=2)
    ref = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb)
    assert got["remote"][0] + got["remote"][1] == _distinct_remote_lines(M, N, K, Gr, Gc, P,
                                                                         placement, ta, tb)
    assert got["remote"][2] == ref["remote"][2]          # C is never cached


def test_misses_nonincreasing_in_ways():
    M, N, K, Gr, Gc, P = 256, 512, 256, 2, 2, 4096
    prev = None
    for ways in (1, 2, 4, 8, 16):
        rec = L.simulate(M, N, K, Gr, Gc, P, "rr", l2_bytes=4 * ways * 128, ways=ways, slots=2)
        m = sum(rec["misses"])
        if prev is not None:
            assert m <= prev
        prev = m


@pytest.mark.parametrize("placement", PLACEMENTS)
def test_cache_never_adds_traffic(placement):
    M, N, K, Gr, Gc, P = 256, 512, 256, 2, 2, 4096
    none = L.simulate(M, N, K, Gr, Gc, P, placement, l2_bytes=0, slots=2)
    some = L.simulate(M, N, K, Gr, Gc, P, placement, l2_bytes=16 * 128 * 4, ways=4, slots=2)
    assert all(s <= n for s, n in zip(some["remote"], none["remote"]))
    assert some["remote"][2] == none["remote"][2]
    assert sum(some["remote_per_chiplet"]) == L.total_remote(some)


@pytest.mark.parametrize("placement", PLACEMENTS)
def test_one_chiplet_is_all_local(placement):
    rec = L.simulate(256, 256, 128, 1, 1, 4096, placement, l2_bytes=64 * 128 * 16, slots=2)
    assert rec["remote"] == [0, 0, 0]
    assert rec["misses"][0] > 0


def test_ccl_keeps_private_operands_local():
    # 1 x 4: B and C are private to their column owner; 4 x 1: A and C.
    r14 = L.simulate(256, 512, 256, 1, 4, 4096, "ccl", l2_bytes=8 * 128 * 16, slots=2)
    assert r14["remote"][1] == 0 and r14["remote"][2] == 0 and r14["remote"][0] > 0
    r41 = L.simulate(512, 256, 256, 4, 1, 4096, "ccl", l2_bytes=8 * 128 * 16, slots=2)
    assert r41["remote"][0] == 0 and r41["remote"][2] == 0 and r41["remote"][1] > 0


def test_partition_tiles_order():
    # 512 x 512 output, 2 x 2 grid: partition 3 holds tiles (2..3, 2..3)
    assert L.partition_tiles(3, 512, 512, 2, 2, "row") == [(2, 2), (2, 3), (3, 2), (3, 3)]
    assert L.partition_tiles(3, 512, 512, 2, 2, "col") == [(2, 2), (3, 2), (2, 3), (3, 3)]


def test_partition_tiles_group_order():
    # 640 x 256 output, one partition: 5 tile rows x 2 tile columns in groups
    # of 2 rows (the last group has 1), each group walked column by column
    assert L.partition_tiles(0, 640, 256, 1, 1, "group", 2) == [
        (0, 0), (1, 0), (0, 1), (1, 1), (2, 0), (3, 0), (2, 1), (3, 1), (4, 0), (4, 1)]
    # partition 1 of a 1 x 2 grid over 640 x 512 holds tile columns 2..3
    assert L.partition_tiles(1, 640, 512, 1, 2, "group", 4) == [
        (0, 2), (1, 2), (2, 2), (3, 2), (0, 3), (1, 3), (2, 3), (3, 3), (4, 2), (4, 3)]
    # one-row groups are the row order; one group of all rows is the column order
    for p in range(4):
        assert L.partition_tiles(p, 1024, 768, 2, 2, "group", 1) == L.partition_tiles(p, 1024, 768, 2, 2, "row")
        assert L.partition_tiles(p, 1024, 768, 2, 2, "group", 4) == L.partition_tiles(p, 1024, 768, 2, 2, "col")
        assert L.partition_tiles(p, 1024, 768, 2, 2, "group", 9) == L.partition_tiles(p, 1024, 768, 2, 2, "col")
    with pytest.raises(ValueError):
        L.partition_tiles(0, 256, 256, 1, 1, "group", 0)


def test_order_grouped_waves_share_panels():
    # M = N = 512, K = 64 (one K step), one chiplet, waves of 4 tiles, a
    # fully associative LRU cache of 4 slices (512 lines; a slice is 128).
    # Grouped (2 rows), worked through access by access:
    #   wave 1 (0,0) (1,0) (0,1) (1,1): A0 A1 B0 B1 miss once each;
    #   wave 2 (0,2) (1,2) (0,3) (1,3): A0 A1 hit, B2 B3 miss;
    #   wave 3 (2,0) (3,0) (2,1) (3,1): A2 A3 B0 B1 miss;
    #   wave 4 (2,2) (3,2) (2,3) (3,3): A2 A3 hit, B2 B3 miss.
    # A misses 4 slices, B misses 8. Row order puts A0 and B0..B3 (5 slices)
    # in one wave, which does not fit, so it misses more B.
    kw = dict(l2_bytes=512 * 128, ways=512, slots=4, k_step=64)
    grp = L.simulate(512, 512, 64, 1, 1, 4096, "rr", traversal="group", group_rows=2, **kw)
    row = L.simulate(512, 512, 64, 1, 1, 4096, "rr", traversal="row", **kw)
    assert grp["misses"] == [4 * 128, 8 * 128]
    assert row["misses"][1] > grp["misses"][1]


# ---------------------------------------------------------------------------
# access order, worked by hand on one chiplet with a fully associative cache
# (row-major operands; an A slice of 128 rows x 64 elements is 128 lines, a
# B slice of 64 rows x 128 columns is 128 lines)
# ---------------------------------------------------------------------------

def _fa(lines):
    return dict(l2_bytes=lines * 128, ways=lines)


def test_order_waves_advance_through_k_together():
    # M=128, N=256, K=128: tiles t0=(0,0), t1=(0,1) share the A panel; two K
    # steps s0, s1. Cache of 384 lines.
    # slots=2: s0: A_s0 miss, B0_s0 miss, A_s0 hit, B1_s0 miss (cache full);
    #          s1: A_s1 miss, B0_s1 miss, A_s1 hit, B1_s1 miss -> A misses 256.
    # slots=1: t0 reads A_s0, B0_s0, A_s1, B0_s1 (A_s0 evicted by the last);
    #          t1 then misses all of A_s0 and A_s1 again -> A misses 512.
    two = L.simulate(128, 256, 128, 1, 1, 4096, "rr", slots=2, **_fa(384))
    one = L.simulate(128, 256, 128, 1, 1, 4096, "rr", slots=1, **_fa(384))
    assert two["misses"] == [256, 512]
    assert one["misses"] == [512, 512]
    assert two["accesses"] == one["accesses"] == [512, 512]


def test_order_traversal():
    # M=N=256, K=64: tiles (0,0) (0,1) (1,0) (1,1); cache of 256 lines holds
    # two slices. Row order re-reads the B panels (A0 A1 stay hot in turn):
    # A misses A0, A1 = 256; B misses B0, B1, B0, B1 = 512. Column order is
    # the mirror image.
    row = L.simulate(256, 256, 64, 1, 1, 4096, "rr", slots=1, traversal="row", **_fa(256))
    col = L.simulate(256, 256, 64, 1, 1, 4096, "rr", slots=1, traversal="col", **_fa(256))
    assert row["misses"] == [256, 512]
    assert col["misses"] == [512, 256]



@pytest.mark.parametrize("placement", PLACEMENTS)
def test_c_read_is_charged_like_the_write(placement):
    M, N, K, Gr, Gc, P = 256, 512, 256, 2, 2, 4096
    ref = T.remote_bytes(M, N, K, Gr, Gc, P, placement, c_read=True)
    got = L.simulate(M, N, K, Gr, Gc, P, placement, l2_bytes=0, slots=2, c_read=True)
    assert got["remote"] == ref["remote"]
    plain = L.simulate(M, N, K, Gr, Gc, P, placement, l2_bytes=4 * 16 * 128, slots=2)
    read = L.simulate(M, N, K, Gr, Gc, P, placement, l2_bytes=4 * 16 * 128, slots=2, c_read=True)
    assert read["remote"][:2] == plain["remote"][:2]
    assert read["remote"][2] == 2 * plain["remote"][2]
    assert read["misses"] == plain["misses"]


@pytest.mark.parametrize("placement", PLACEMENTS)
@pytest.mark.parametrize("e,k_step", [((1, 1, 2), 128), ((1, 1, 4), 128), ((2, 2, 4), 64),
                                      ((4, 4, 4), 32)])
def test_element_sizes_capacity_zero_is_tile_charge(placement, e, k_step):
    """With a K step of one line per row (128 / e_A elements) the no-cache
    limit still equals the tile-charge model for every element size."""
    M, N, K, Gr, Gc, P = 256, 512, 512, 2, 2, 4096
    ref = T.remote_bytes(M, N, K, Gr, Gc, P, placement, 1, 0, e=e)
    got = L.simulate(M, N, K, Gr, Gc, P, placement, 1, 0, l2_bytes=0, slots=2, k_step=k_step, e=e)
    assert got["remote"] == ref["remote"]
