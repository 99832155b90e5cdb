"""Partition rules of a CCL GEMM: grid validity, tile ownership, grid choice.

Sec. II-B: the output C is split into 128x128 tiles, one CTA per tile; a
locality-aware scheduler runs each tile on the chiplet that owns it.
Sec. III-A: C is partitioned among the chiplets, and A and B are laid out so
that the owning chiplet also holds the operand regions its tiles read.
Sec. IV-A "Hardware Configuration": 128x128 output tiles.

Readings (the paper does not write these out):
  * A grid "Gr x Gc" splits M into Gr row blocks and N into Gc column blocks;
    partition p = pr * Gc + pc is chiplet p.
  * A is split by the same grid over its own (rows, cols) = (M, K), B over
    (K, N): A along K by Gc, B along K by Gr (Sec. III-C says CCL applies to
    A, B and C, but the paper only writes the map for B split along N).
  * Partitions must be tile-aligned: M % (Gr*128) == 0, N % (Gc*128) == 0,
    K % Gr == 0 and K % Gc == 0.
  * Per-GEMM choice of coarse vs fine partitioning (Sec. IV-A "Baselines"):
    the automatic grid minimises the CCL remote bytes (which equal the
    floor); ties go to the grid whose shared operands replicate fewer bytes
    (Fig. 2(b): the shared operand is the one that lives in every sharer's
    L2), then to the smaller Gr.
  * Chiplet c of G maps to XCDs c*(8/G) ... c*(8/G) + 8/G - 1 (Sec. IV-A: a
    locality domain is a group of XCDs; MI355X has 8 XCDs).
"""
from __future__ import annotations

TILE = 128          # model output tile, Sec. IV-A
ELEM_BYTES = 2      # bf16 (Sec. IV-A: BF16 GEMMs)
N_XCD = 8


def elem_sizes(e) -> tuple[int, int, int]:
    """Element bytes of (A, B, C): one int for all three, or a 3-tuple
    (Fig. 7 sweeps the data type; fp8 operands with a bf16 or fp32 output
    give different sizes per operand)."""
    if isinstance(e, (tuple, list)):
        ea, eb, ec = e
        return int(ea), int(eb), int(ec)
    return int(e), int(e), int(e)


def is_pow2(x: int) -> bool:
    return x > 0 and (x & (x - 1)) == 0


def grid_valid(M: int, N: int, K: int, G: int, Gr: int) -> bool:
    """True iff the Gr x (G/Gr) grid gives tile-aligned partitions."""
    if Gr <= 0 or G % Gr != 0:
        return False
    Gc = G // Gr
    return (M % (Gr * TILE) == 0 and N % (Gc * TILE) == 0
            and K % Gr == 0 and K % Gc == 0)


def owner(ti: int, tj: int, M: int, N: int, Gr: int, Gc: int) -> int:
    """Chiplet that owns output tile (ti, tj) (128x128 tiles)."""
    tiles_r = M // (Gr * TILE)      # tile rows per partition
    tiles_c = N // (Gc * TILE)
    return (ti // tiles_r) * Gc + (tj // tiles_c)


def floor_bytes(M: int, N: int, K: int, Gr: int, Gc: int, e=ELEM_BYTES) -> int:
    """Lower bound on remote bytes of any layout under this ownership.

    Each A element is read by the Gc chiplets of its grid row, N/(Gc*128)
    times by each; at most one of them holds it, so (Gc-1)/Gc of its reads are
    remote. Same for B with Gr. C writes can all be local.
    Integer form of e*M*N*K*[(Gc-1)/(Gc*128) + (Gr-1)/(Gr*128)] (with e_A
    and e_B for the two terms when the operands differ in size).
    """
    ea, eb, _ = elem_sizes(e)
    a = ea * M * K * (N // (Gc * TILE)) * (Gc - 1)
    b = eb * K * N * (M // (Gr * TILE)) * (Gr - 1)
    return a + b


def shared_replica_bytes(M: int, N: int, K: int, Gr: int, Gc: int, e=ELEM_BYTES) -> float:
    """Bytes of each shared operand that its non-owning sharers also need."""
    ea, eb, _ = elem_sizes(e)
    return ea * M * K * (Gc - 1) / Gc + eb * K * N * (Gr - 1) / Gr


def auto_grid_rows(M: int, N: int, K: int, G: int, e=ELEM_BYTES) -> int:
    """Grid chosen for grid_rows = 0; 0 if no tile-aligned grid exists."""
    best = None
    for Gr in range(1, G + 1):
        if not grid_valid(M, N, K, G, Gr):
            continue
        Gc = G // Gr
        key = (floor_bytes(M, N, K, Gr, Gc, e), shared_replica_bytes(M, N, K, Gr, Gc, e), Gr)
        if best is None or key < best[0]:
            best = (key, Gr)
    return 0 if best is None else best[1]


def xcds_of_chiplet(c: int, G: int) -> list[int]:
    per = N_XCD // G
    return list(range(c * per, c * per + per))
