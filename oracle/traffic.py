"""Integer remote-HBM-byte model (tile charge, no cache), Sec. IV-A.

What is charged (Sec. II-B, Sec. IV-A "Metrics"):
  * output tile (ti, tj) of 128x128 (Sec. IV-A) runs on its owning chiplet
    (see plan.owner);
  * it reads A[ti*128 : +128, 0:K] and B[0:K, tj*128 : +128] and writes
    C[ti*128 : +128, tj*128 : +128];
  * each element access costs e bytes and is remote iff the chiplet holding
    the element's page differs from the tile's owner. Remote reads and
    remote output writes both count.

Where each element's page lives (the three placements of Sec. IV-A
"Baselines"); s is the element's byte offset in the STORED tensor, which is
row-major, or row-major of the transpose when the operand is stored
transposed (e.g. A = H^T held as H):
  RR(P)      consecutive P-byte pages go to chiplets in address order:
             chip = floor(s / P) mod G  (each tensor is its own allocation,
             aligned so that its page 0 is on chiplet 0);
  COARSE(P)  G large contiguous page-granular chunks, chunk g on chiplet g:
             n_p = ceil(bytes / P), chip = floor(floor(s / P) * G / n_p);
  CCL(P)     the operand is stored in CCL with strips padded to P, and every
             page of strip b is placed on chiplet b: chip = block b(r, c).

With beta != 0 (C = alpha A B + beta C, Sec. II-B), the C tile is also read
by its owner; the paper notes that this read is partitioned exactly like the
write, so it is charged like the write (c_read=True doubles the C terms).

Readings (the paper simulates per-chiplet L2 caches; this model has none, so
it charges every tile's full panel reads; its ratios are not the paper's):
  see the notes at each function.

The result of remote_bytes() is computed with per-panel chiplet histograms.
Pinned by: an element-by-element brute force on small shapes (tests), the
closed forms floor / accessed, CCL == floor, G == 1 => 0, and special cases
where RR or COARSE coincide with the CCL blocks.
"""
from __future__ import annotations

import numpy as np

from . import layout
from .plan import TILE, elem_sizes, owner, floor_bytes

RR, COARSE, CCL = "rr", "coarse", "ccl"
PLACEMENTS = (RR, COARSE, CCL)
OPS = ("A", "B", "C")


def stored_offset(r, c, R, Cc, trans, e=2):
    """Byte offset of logical (r, c) in the stored row-major tensor."""
    r = np.asarray(r, dtype=np.int64)
    c = np.asarray(c, dtype=np.int64)
    if trans:
        return (c * R + r) * e          # stored tensor is Cc x R
    return (r * Cc + c) * e


def chip_of(r, c, R, Cc, trans, placement, Pr, Pc, P, e=2):
    """Chiplet holding logical element (r, c) of an R x Cc operand."""
    G = Pr * Pc
    if placement == CCL:
        return layout.block_of(r, c, R, Cc, Pr, Pc)
    page = stored_offset(r, c, R, Cc, trans, e) // P
    if placement == RR:
        return page % G
    if placement == COARSE:
        n_pages = -(-(R * Cc * e) // P)
        return (page * G) // n_pages
    raise ValueError(placement)


def _hist(chips: np.ndarray, G: int) -> np.ndarray:
    return np.bincount(chips.reshape(-1), minlength=G).astype(np.int64)


def remote_bytes(M, N, K, Gr, Gc, P, placement, trans_a=0, trans_b=0, e=2, c_read=False):
    """Remote bytes of C = A B (or alpha A B + beta C with c_read) under one placement.

    e: element bytes, one for all operands or (e_A, e_B, e_C).

    Returns a dict of Python ints:
      accessed[A,B,C], remote[A,B,C], remote_per_chiplet[G],
      floor, footprint[A,B,C] (bytes of each stored operand, padding included).
    """
    G = Gr * Gc
    ea, eb, ec = elem_sizes(e)
    TM, TN = M // TILE, N // TILE
    own = np.array([[owner(ti, tj, M, N, Gr, Gc) for tj in range(TN)] for ti in range(TM)],
                   dtype=np.int64)
    remote = {"A": 0, "B": 0, "C": 0}
    per_chip = np.zeros(G, dtype=np.int64)

    # A row panels: panel ti holds TILE*K elements; every tile in row ti reads it.
    cols = np.arange(K)
    for ti in range(TM):
        rows = np.arange(ti * TILE, (ti + 1) * TILE)
        h = _hist(chip_of(rows[:, None], cols[None, :], M, K, trans_a, placement, Gr, Gc, P, ea), G)
        for tj in range(TN):
            o = own[ti, tj]
            rb = ea * (TILE * K - int(h[o]))
            remote["A"] += rb
            per_chip[o] += rb
    # B column panels: panel tj holds K*TILE elements; every tile in column tj reads it.
    rows = np.arange(K)
    for tj in range(TN):
        cols = np.arange(tj * TILE, (tj + 1) * TILE)
        h = _hist(chip_of(rows[:, None], cols[None, :], K, N, trans_b, placement, Gr, Gc, P, eb), G)
        for ti in range(TM):
            o = own[ti, tj]
            rb = eb * (K * TILE - int(h[o]))
            remote["B"] += rb
            per_chip[o] += rb
    # C tiles: each written once by its owner (C is never stored transposed),
    # and read once before that when c_read.
    c_times = 2 if c_read else 1
    cols = np.arange(N)
    for ti in range(TM):
        rows = np.arange(ti * TILE, (ti + 1) * TILE)
        ch = chip_of(rows[:, None], cols[None, :], M, N, 0, placement, Gr, Gc, P, ec)
        ch = ch.reshape(TILE, TN, TILE).transpose(1, 0, 2).reshape(TN, -1)
        for tj in range(TN):
            o = own[ti, tj]
            rb = c_times * ec * int(np.count_nonzero(ch[tj] != o))
            remote["C"] += rb
            per_chip[o] += rb

    accessed = {"A": ea * M * K * TN, "B": eb * K * N * TM, "C": c_times * ec * M * N}
    esz = {"A": ea, "B": eb, "C": ec}
    if placement == CCL:
        fp = {op: layout.total_bytes(*layout.operand_shape(op, M, N, K), Gr, Gc, P, esz[op]) for op in OPS}
    else:
        fp = {op: esz[op] * int(np.prod(layout.operand_shape(op, M, N, K))) for op in OPS}
    return {
        "accessed": [accessed[o] for o in OPS],
        "remote": [int(remote[o]) for o in OPS],
        "remote_per_chiplet": [int(x) for x in per_chip],
        "floor": floor_bytes(M, N, K, Gr, Gc, e),
        "footprint": [int(fp[o]) for o in OPS],
    }


def total_remote(rec) -> int:
    return int(sum(rec["remote"]))
