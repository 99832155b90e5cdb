"""Pins of partition validity, ownership and the automatic grid choice."""
from fractions import Fraction

import pytest

from oracle import plan as PL


def test_grid_validity_definition():
    # tile-aligned partitions only (128x128 model tiles, Sec. IV-A)
    assert PL.grid_valid(256, 512, 256, 4, 2)
    assert not PL.grid_valid(256, 512, 256, 4, 4)      # 256 rows / 4 < 128
    assert not PL.grid_valid(256, 512, 255, 4, 2)      # K not divisible
    assert not PL.grid_valid(256, 512, 256, 4, 3)      # 3 does not divide 4
    valid = [g for g in (1, 2, 4, 8) if PL.grid_valid(768, 2048, 4096, 8, g)]
    assert valid == [1, 2]
    valid = [g for g in (1, 2, 4, 8) if PL.grid_valid(4096, 768, 2048, 8, g)]
    assert valid == [4, 8]


@pytest.mark.parametrize("M,N,Gr,Gc", [(256, 512, 2, 2), (1024, 2048, 2, 4), (768, 2048, 1, 8), (4096, 768, 8, 1)])
def test_owner_partitions_tiles_evenly_into_rectangles(M, N, Gr, Gc):
    TM, TN = M // 128, N // 128
    counts = [0] * (Gr * Gc)
    for ti in range(TM):
        for tj in range(TN):
            o = PL.owner(ti, tj, M, N, Gr, Gc)
            counts[o] += 1
            # partition (pr, pc) is the rectangle of rows pr*M/Gr.., cols pc*N/Gc..
            assert o == (ti * 128 // (M // Gr)) * Gc + (tj * 128 // (N // Gc))
    assert len(set(counts)) == 1 and sum(counts) == TM * TN


def test_floor_ratio_between_grids():
    """floor is e MNK [(Gc-1)/Gc + (Gr-1)/Gr] / 128: 2x4 vs 1x8 is
    (3/4 + 1/2) / (7/8) = 10/7."""
    a = PL.floor_bytes(768, 2048, 4096, 2, 4)
    b = PL.floor_bytes(768, 2048, 4096, 1, 8)
    assert Fraction(a, b) == Fraction(10, 7)


def test_auto_grid_choices():
    # Qwen backward: dW_down (768x2048x4096) -> 1x8, dH (4096x768x2048) -> 8x1
    assert PL.auto_grid_rows(768, 2048, 4096, 8) == 1
    assert PL.auto_grid_rows(4096, 768, 2048, 8) == 8
    # 1xG and Gx1 tie on the floor; the smaller shared operand wins:
    # 1x8 shares A (M x K), 8x1 shares B (K x N)
    assert PL.auto_grid_rows(1024, 4096, 1024, 8) == 1      # A smaller than B
    assert PL.auto_grid_rows(4096, 1024, 1024, 8) == 8      # B smaller than A
    assert PL.auto_grid_rows(1024, 1024, 1024, 8) == 1      # full tie -> smaller Gr
    assert PL.auto_grid_rows(100, 100, 100, 8) == 0         # nothing aligned


def test_chiplet_to_xcd_map():
    assert PL.xcds_of_chiplet(3, 8) == [3]
    assert PL.xcds_of_chiplet(1, 4) == [2, 3]
    assert PL.xcds_of_chiplet(0, 1) == list(range(8))
