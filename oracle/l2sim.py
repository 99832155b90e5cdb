"""Finite-L2 remote-HBM-traffic model (Sec. IV-A "Simulation framework",
"Hardware Configuration", "Metrics"; Fig. 7 capacity sweep).

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper's simulator does (Sec. IV-A): CTAs, one per 128x128 output
tile, run on the chiplet that owns their tile and issue operand accesses in
the order given by the GEMM shape and the CTA traversal; each chiplet has a
private L2 (the paper: 8 MB, 128-byte lines, 16-way); an L2 miss goes to
HBM and is remote when the line's page lives on another chiplet; writes
of output to another chiplet's memory also count.

The paper does not write out the access order, the set index or the
replacement policy. Readings taken here (each one a parameter or a stated
convention, identical in the library's implementation):
  * Execution: chiplet p runs the tiles of its partition in traversal order
    ("row": tile rows outer; "col": tile columns outer), `slots` tiles at a
    time. The tiles of one such wave advance through K together, k_step
    elements of K at a time: at step s every tile of the wave, in wave
    order, reads its A slice (128 rows x k_step) and then its B slice
    (k_step x 128 columns). When the wave has finished K, each of its tiles
    writes its C tile. Chiplets have private caches, so the interleaving of
    different chiplets does not matter.
  * A slice is read as the distinct 128-byte lines it touches in its STORED
    layout (row-major, row-major of the transpose, or CCL), in increasing
    address order; each line is one L2 access.
  * Addresses: A at byte 0, B at 2^40, C at 2^41 (separate allocations, far
    apart). Line number = address // line.
  * Set index: the line number folded by XOR into log2(sets) bits (a hashed
    index, as GPU L2s use; plain modulo indexing would map the 128 rows of a
    power-of-two-strided panel onto a few sets). sets = capacity / (line *
    ways), a power of two.
  * Replacement: true LRU within a set. Capacity 0 means no cache: every
    access misses.
  * A line's home chiplet is the chiplet of its first byte under the
    placement (same placements as the tile-charge model: RR, COARSE, CCL).
    A miss is remote when home != the tile's owner; remote bytes are
    misses * line.
  * C is written once per tile and is not allocated in L2 (the paper counts
    output writes to another chiplet separately from read misses); a C line
    whose home is not the owner costs line bytes. With beta != 0 (c_read)
    the tile's C lines are also read once, the same way, before the write.

Pinned by (tests/test_oracle_l2sim.py): hand-worked LRU sequences; the
LRU core against an independent reuse-distance computation; capacity 0
equal to the tile-charge model; an unbounded cache equal to each chiplet's
distinct remote lines; misses non-increasing in associativity; G = 1 gives
zero.
"""
from __future__ import annotations

import numpy as np

from . import layout
from .plan import TILE, elem_sizes, owner

RR, COARSE, CCL = "rr", "coarse", "ccl"
OPS = ("A", "B", "C")
BASE = {"A": 0, "B": 1 << 40, "C": 1 << 41}


def fold_set(line: int, sets: int) -> int:
    """Set of a line: XOR of the line number's log2(sets)-bit chunks."""
    if sets == 1:
        return 0
    bits = sets.bit_length() - 1
    x = 0
    while line:
        x ^= line & (sets - 1)
        line >>= bits
    return x


class LRUCache:
    """Set-associative LRU cache of line numbers. capacity 0 = no cache."""

    def __init__(self, capacity_bytes: int, ways: int, line: int):
        self.off = capacity_bytes == 0
        if not self.off:
            if capacity_bytes % (line * ways):
                raise ValueError("capacity is not a whole number of sets")
            self.sets = capacity_bytes // (line * ways)
            if self.sets & (self.sets - 1):
                raise ValueError("number of sets must be a power of two")
            self.ways = ways
            self.lists = [[] for _ in range(self.sets)]   # index 0 = most recent

    def access(self, ln: int) -> bool:
        """Touch line ln; True on a hit."""
        if self.off:
            return False
        lst = self.lists[fold_set(ln, self.sets)]
        if ln in lst:
            lst.remove(ln)
            lst.insert(0, ln)
            return True
        lst.insert(0, ln)
        if len(lst) > self.ways:
            lst.pop()
        return False


def _stored_offsets(op, rows, cols, M, N, K, Gr, Gc, P, placement, trans, e):
    """Byte offsets (in the operand's own buffer) of the logical elements
    rows x cols of operand op, as stored under the placement."""
    R, Cc = layout.operand_shape(op, M, N, K)
    r = np.asarray(rows, dtype=np.int64)[:, None]
    c = np.asarray(cols, dtype=np.int64)[None, :]
    if placement == CCL:
        return layout.ccl_offset(r, c, R, Cc, Gr, Gc, P, e)
    if trans:
        return (c * R + r) * e
    return (r * Cc + c) * e


def _home(op, off, M, N, K, Gr, Gc, P, placement, e):
    """Chiplet holding the byte at offset `off` of operand op's buffer."""
    G = Gr * Gc
    R, Cc = layout.operand_shape(op, M, N, K)
    if placement == CCL:
        return off // layout.strip_stride_bytes(R, Cc, Gr, Gc, P, e)
    page = off // P
    if placement == RR:
        return page % G
    if placement == COARSE:
        n_pages = -(-(R * Cc * e) // P)
        return page * G // n_pages
    raise ValueError(placement)


def _slice_lines(op, rows, cols, M, N, K, Gr, Gc, P, placement, trans, e, line):
    """Distinct lines a slice touches, ascending, with each line's home."""
    off = _stored_offsets(op, rows, cols, M, N, K, Gr, Gc, P, placement, trans, e).reshape(-1)
    line_off = np.unique(off // line) * line          # offsets of the lines' first bytes
    lines = (BASE[op] + line_off) // line
    homes = _home(op, line_off, M, N, K, Gr, Gc, P, placement, e)
    return [int(x) for x in lines], [int(h) for h in homes]


def partition_tiles(p, M, N, Gr, Gc, traversal, group_rows=0):
    """Tiles (ti, tj) of partition p in traversal order: "row" (tile rows
    outer), "col" (tile columns outer) or "group" (the partition's tile rows
    cut into groups of group_rows, the last one shorter if needed; the
    groups in order, each walked column by column down its rows)."""
    TR, TC = M // (Gr * TILE), N // (Gc * TILE)
    pr, pc = p // Gc, p % Gc
    rows = range(pr * TR, (pr + 1) * TR)
    cols = range(pc * TC, (pc + 1) * TC)
    if traversal == "row":
        return [(ti, tj) for ti in rows for tj in cols]
    if traversal == "col":
        return [(ti, tj) for tj in cols for ti in rows]
    if traversal == "group":
        if group_rows < 1:
            raise ValueError(group_rows)
        out = []
        for g0 in range(0, TR, group_rows):
            grp = rows[g0:g0 + group_rows]
            out += [(ti, tj) for tj in cols for ti in grp]
        return out
    raise ValueError(traversal)


def simulate(M, N, K, Gr, Gc, P, placement, trans_a=0, trans_b=0, *,
             l2_bytes, slots, ways=16, line=128, k_step=64, traversal="row", e=2,
             c_read=False, group_rows=0):
    """Remote-HBM traffic of C = A B with a private L2 per chiplet.

    Returns a dict of Python ints:
      accesses[A, B]  line accesses issued
      misses[A, B]    of which missed
      remote[A, B, C] bytes: remote misses * line (A, B), remote C line writes
      remote_per_chiplet[G]  charged to the chiplet running the tile
    e: element bytes, one for all operands or (e_A, e_B, e_C).
    """
    G = Gr * Gc
    ea, eb, ec = elem_sizes(e)
    esz = {"A": ea, "B": eb, "C": ec}
    nk = -(-K // k_step)
    acc = {"A": 0, "B": 0}
    mis = {"A": 0, "B": 0}
    rem = {"A": 0, "B": 0, "C": 0}
    per_chip = [0] * G
    trans = {"A": trans_a, "B": trans_b, "C": 0}
    for p in range(G):
        cache = LRUCache(l2_bytes, ways, line)
        tiles = partition_tiles(p, M, N, Gr, Gc, traversal, group_rows)
        for w0 in range(0, len(tiles), slots):
            wave = tiles[w0:w0 + slots]
            for s in range(nk):
                ks = range(s * k_step, min(K, (s + 1) * k_step))
                for ti, tj in wave:
                    assert owner(ti, tj, M, N, Gr, Gc) == p
                    m = range(ti * TILE, (ti + 1) * TILE)
                    n = range(tj * TILE, (tj + 1) * TILE)
                    for op, rows, cols in (("A", m, ks), ("B", ks, n)):
                        lines, homes = _slice_lines(op, rows, cols, M, N, K, Gr, Gc, P,
                                                    placement, trans[op], esz[op], line)
                        for ln, h in zip(lines, homes):
                            acc[op] += 1
                            if not cache.access(ln):
                                mis[op] += 1
                                if h != p:
                                    rem[op] += line
                                    per_chip[p] += line
            for ti, tj in wave:
                lines, homes = _slice_lines("C", range(ti * TILE, (ti + 1) * TILE),
                                            range(tj * TILE, (tj + 1) * TILE),
                                            M, N, K, Gr, Gc, P, placement, 0, ec, line)
                for h in homes:
                    if h != p:
                        for _ in range(2 if c_read else 1):
                            rem["C"] += line
                            per_chip[p] += line
    return {
        "accesses": [acc["A"], acc["B"]],
        "misses": [mis["A"], mis["B"]],
        "remote": [rem[o] for o in OPS],
        "remote_per_chiplet": per_chip,
    }


def total_remote(rec) -> int:
    return int(sum(rec["remote"]))
