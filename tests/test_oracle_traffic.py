"""Pins of the oracle's remote-byte model (Sec. IV-A placements and metric).

The oracle aggregates per-panel chiplet histograms. These tests check it
against (1) a brute force that materialises every stored byte address and
walks each tile's accesses, (2) the closed forms for accessed bytes and the
floor, (3) special cases where round-robin or coarse placement provably puts
every element on its CCL block's chiplet, and (4) conservation / symmetry.
"""
import math

import numpy as np
import pytest

from oracle import traffic as T
from oracle import plan as PL


# ---------------------------------------------------------------------------
# brute force: explicit per-element page table, per-tile access walk
# ---------------------------------------------------------------------------

def _stored_addresses(R, Cc, trans, e=2):
    """Byte address of every logical element, by materialising the stored
    tensor (row-major, or row-major of the transpose) as an index array."""
    if trans:
        return np.arange(R * Cc, dtype=np.int64).reshape(Cc, R).T * e
    return np.arange(R * Cc, dtype=np.int64).reshape(R, Cc) * e


def _page_table(n_pages, G, placement):
    """Chiplet of each page, built by walking the pages in address order."""
    table = np.empty(n_pages, dtype=np.int64)
    if placement == "rr":
        chip = 0
        for p in range(n_pages):          # consecutive pages to chiplets in turn
            table[p] = chip
            chip = (chip + 1) % G
    else:
        # G contiguous chunks; chunk g starts at the first page p with
        # p * G >= g * n_pages (so chunk g = pages [ceil(g n / G), ceil((g+1) n / G)))
        bounds = [-(-(g * n_pages) // G) for g in range(G + 1)]
        for g in range(G):
            table[bounds[g]:bounds[g + 1]] = g
    return table


def _chip_matrix(R, Cc, trans, placement, Gr, Gc, P, e=2):
    G = Gr * Gc
    if placement == "ccl":
        m = np.empty((R, Cc), dtype=np.int64)
        hr, wc = R // Gr, Cc // Gc
        for pr in range(Gr):
            for pc in range(Gc):
                m[pr * hr:(pr + 1) * hr, pc * wc:(pc + 1) * wc] = pr * Gc + pc
        return m
    addr = _stored_addresses(R, Cc, trans, e)
    n_pages = -(-(R * Cc * e) // P)
    return _page_table(n_pages, G, placement)[addr // P]


def brute_remote(M, N, K, Gr, Gc, P, placement, ta=0, tb=0, chips=None, e=2, c_read=False):
    G = Gr * Gc
    es = e if isinstance(e, tuple) else (e, e, e)
    if chips is None:
        chips = (_chip_matrix(M, K, ta, placement, Gr, Gc, P, es[0]),
                 _chip_matrix(K, N, tb, placement, Gr, Gc, P, es[1]),
                 _chip_matrix(M, N, 0, placement, Gr, Gc, P, es[2]))
    chA, chB, chC = chips
    remote = [0, 0, 0]
    accessed = [0, 0, 0]
    per = [0] * G
    rows_per_part, cols_per_part = M // Gr, N // Gc
    for m0 in range(0, M, 128):
        for n0 in range(0, N, 128):
            own = (m0 // rows_per_part) * Gc + (n0 // cols_per_part)
            blocks = [(0, chA[m0:m0 + 128, :]), (1, chB[:, n0:n0 + 128]),
                      (2, chC[m0:m0 + 128, n0:n0 + 128])]
            if c_read:                          # beta != 0: the C tile is read too
                blocks.append((2, chC[m0:m0 + 128, n0:n0 + 128]))
            for i, blk in blocks:
                nb = es[i] * int(np.count_nonzero(blk != own))
                remote[i] += nb
                accessed[i] += es[i] * blk.size
                per[own] += nb
    return remote, accessed, per


CASES = [
    # M, N, K, Gr, Gc, P, ta, tb
    (256, 512, 256, 2, 2, 4096, 0, 0),
    (256, 512, 256, 2, 2, 256, 0, 0),
    (256, 512, 256, 2, 2, 65536, 0, 0),
    (256, 256, 384, 1, 2, 4096, 1, 0),
    (256, 256, 384, 2, 1, 1024, 0, 1),
    (512, 256, 192, 4, 1, 512, 1, 1),
    (256, 1024, 96, 1, 8, 128, 0, 0),
    (1024, 256, 320, 8, 1, 4096, 0, 1),
    (384, 768, 201, 1, 3, 2048, 1, 0),
    (128, 128, 64, 1, 1, 4096, 0, 0),
]


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", CASES)
@pytest.mark.parametrize("placement", T.PLACEMENTS)
def test_histogram_model_equals_brute_force(M, N, K, Gr, Gc, P, ta, tb, placement):
    rec = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb)
    remote, accessed, per = brute_remote(M, N, K, Gr, Gc, P, placement, ta, tb)
    assert rec["remote"] == remote
    assert rec["accessed"] == accessed
    assert rec["remote_per_chiplet"] == per


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", CASES[:5])
@pytest.mark.parametrize("placement", T.PLACEMENTS)
def test_c_read_equals_brute_force(M, N, K, Gr, Gc, P, ta, tb, placement):
    rec = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb, c_read=True)
    remote, accessed, per = brute_remote(M, N, K, Gr, Gc, P, placement, ta, tb, c_read=True)
    assert rec["remote"] == remote
    assert rec["accessed"] == accessed
    assert rec["remote_per_chiplet"] == per
    assert rec["accessed"][2] == 2 * 2 * M * N


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", CASES[:6])
@pytest.mark.parametrize("placement", T.PLACEMENTS)
@pytest.mark.parametrize("e", [(1, 1, 2), (1, 1, 4), (2, 2, 4), (4, 4, 4)])
def test_element_sizes_equal_brute_force(M, N, K, Gr, Gc, P, ta, tb, placement, e):
    """fp8 / bf16 / fp32 operands (Fig. 7 data-type sweep): the page an
    element lands on depends on its byte size."""
    rec = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb, e=e)
    remote, accessed, per = brute_remote(M, N, K, Gr, Gc, P, placement, ta, tb, e=e)
    assert rec["remote"] == remote
    assert rec["accessed"] == accessed
    assert rec["remote_per_chiplet"] == per
    if placement == "ccl":
        ea, eb, _ = e
        assert sum(rec["remote"]) == rec["floor"] == round(
            M * N * K * (ea * (Gc - 1) / (Gc * 128) + eb * (Gr - 1) / (Gr * 128)))


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", CASES)
def test_closed_forms(M, N, K, Gr, Gc, P, ta, tb):
    """accessed = e (MNK/BN + MNK/BM + MN); CCL remote = floor
    = e MNK [(Gc-1)/(Gc BN) + (Gr-1)/(Gr BM)]; CCL never writes C remotely;
    each chiplet carries floor/G."""
    e, G = 2, Gr * Gc
    rec = T.remote_bytes(M, N, K, Gr, Gc, P, "ccl", ta, tb)
    assert sum(rec["accessed"]) == e * (M * N * K // 128 + M * N * K // 128 + M * N)
    fl = e * M * N * K * ((Gc - 1) / (Gc * 128) + (Gr - 1) / (Gr * 128))
    assert rec["floor"] == round(fl)
    assert sum(rec["remote"]) == rec["floor"]
    assert rec["remote"][2] == 0
    assert (rec["remote"][0] == 0) == (Gc == 1)
    assert (rec["remote"][1] == 0) == (Gr == 1)
    assert all(x * G == rec["floor"] for x in rec["remote_per_chiplet"])


@pytest.mark.parametrize("M,N,K,Gr,Gc,P,ta,tb", CASES[:6])
@pytest.mark.parametrize("placement", ("rr", "coarse"))
def test_floor_is_lower_bound_and_conservation(M, N, K, Gr, Gc, P, ta, tb, placement):
    rec = T.remote_bytes(M, N, K, Gr, Gc, P, placement, ta, tb)
    assert sum(rec["remote"]) >= rec["floor"]
    assert sum(rec["remote_per_chiplet"]) == sum(rec["remote"])
    for r, a in zip(rec["remote"], rec["accessed"]):
        assert 0 <= r <= a


def test_floor_bounds_arbitrary_placements():
    """No page placement at all beats the floor: random chiplet assignments
    of every element (finer than any page) stay above it."""
    rng = np.random.default_rng(5)
    M, N, K, Gr, Gc = 256, 512, 64, 2, 2
    fl = PL.floor_bytes(M, N, K, Gr, Gc)
    for _ in range(5):
        chips = tuple(rng.integers(0, 4, size=s) for s in ((M, K), (K, N), (M, N)))
        remote, _, _ = brute_remote(M, N, K, Gr, Gc, 4096, "rr", chips=chips)
        assert sum(remote) >= fl


@pytest.mark.parametrize("M,N,K,trans", [(256, 128, 64, 0), (128, 256, 320, 1)])
@pytest.mark.parametrize("P", [128, 4096, 65536])
def test_single_chiplet_has_no_remote_bytes(M, N, K, trans, P):
    for pl in T.PLACEMENTS:
        rec = T.remote_bytes(M, N, K, 1, 1, P, pl, trans, trans)
        assert rec["remote"] == [0, 0, 0] and rec["floor"] == 0


@pytest.mark.parametrize("G,P", [(2, 512), (4, 256), (8, 256)])
def test_rr_equals_ccl_when_slice_is_one_page(G, P):
    """1 x G grid with rows of exactly G pages (N e = K e = G P): the
    round-robin page order puts every row slice on its CCL chiplet, so RR
    reaches the floor (Sec. II-B: misalignment is what makes RR remote)."""
    N = K = G * P // 2
    M = 256
    rr = T.remote_bytes(M, N, K, 1, G, P, "rr")
    ccl = T.remote_bytes(M, N, K, 1, G, P, "ccl")
    assert rr["remote"] == ccl["remote"]
    # one page per slice -> a shifted phase breaks it: RR with page P/2 is worse
    rr_half = T.remote_bytes(M, N, K, 1, G, P // 2, "rr")
    assert sum(rr_half["remote"]) > sum(ccl["remote"])


@pytest.mark.parametrize("M,N,K,G", [(1024, 256, 512, 8), (512, 384, 256, 4), (256, 128, 64, 2)])
def test_coarse_equals_ccl_on_row_block_grid(M, N, K, G):
    """G x 1 grid, row-major operands with page-aligned row blocks: coarse
    chunks are exactly the CCL row blocks (Sec. IV-A: coarse-optimal GEMMs)."""
    P = 256
    co = T.remote_bytes(M, N, K, G, 1, P, "coarse")
    ccl = T.remote_bytes(M, N, K, G, 1, P, "ccl")
    assert co["remote"] == ccl["remote"]


def test_tiny_workload_values():
    """tiny workload (256x512x256, 2x2, 4 KB): brute force reproduces the
    model's per-operand values; CCL = floor; RR > COARSE > CCL."""
    vals = {}
    for pl in T.PLACEMENTS:
        rec = T.remote_bytes(256, 512, 256, 2, 2, 4096, pl)
        remote, _, _ = brute_remote(256, 512, 256, 2, 2, 4096, pl)
        assert rec["remote"] == remote
        vals[pl] = sum(remote)
    assert vals["rr"] > vals["coarse"] > vals["ccl"] == PL.floor_bytes(256, 512, 256, 2, 2)
    assert math.isclose(vals["ccl"], 524288)
