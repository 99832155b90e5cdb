"""Pins of the oracle's CCL address map (Sec. III-A, III-B Eq. 1-3, III-C).

Everything here runs on the CPU. The checks come from outside the oracle's
own block formula: the paper's Eq. 3 as printed, the CuTe stride view of
Sec. III-C realised with numpy's stride machinery, the numbers printed in the
text (tests/golden/paper_values.json), and structural properties.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import layout as L

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _runs(seq):
    return [len(list(g)) for _, g in itertools.groupby(seq)]


@pytest.mark.parametrize("K,N,G", [(4, 8, 2), (16, 64, 4), (7, 24, 3), (32, 256, 8)])
def test_block_map_reduces_to_eq3(K, N, G):
    """Pr = 1, Pc = G, page = element size (no padding): offset/e == Eq. 3."""
    k, n = np.meshgrid(np.arange(K), np.arange(N), indexing="ij")
    off = L.ccl_offset(k, n, K, N, 1, G, P=2, e=2)
    w = N // G
    # Eq. 1 and Eq. 3 spelled out directly
    expect = (n // w) * K * w + k * w + (n % w)
    assert np.array_equal(off // 2, expect)
    assert np.array_equal(L.eq3_index(k, n, K, N, G), expect)


@pytest.mark.parametrize("K,N,G", [(4, 8, 2), (16, 64, 4), (32, 256, 8)])
def test_pack_matches_cute_stride_view(K, N, G):
    """Sec. III-C: the CCL buffer viewed as (K, G, N/G) with strides
    (w, K*w, 1) (in elements) is the logical matrix reshaped to (K, G, w)."""
    rng = np.random.default_rng(0)
    B = rng.integers(0, 65535, size=(K, N), dtype=np.uint16)
    buf = L.pack(B, 1, G, P=2)
    w = N // G
    it = buf.itemsize
    view = np.lib.stride_tricks.as_strided(buf, shape=(K, G, w), strides=(w * it, K * w * it, it))
    assert np.array_equal(view, B.reshape(K, G, w))


@pytest.mark.parametrize("K,N,G", [(4, 8, 2), (16, 64, 4), (7, 24, 3), (32, 256, 8)])
def test_cute_index_is_eq3_and_the_stride_view(K, N, G):
    """Sec. III-C's coordinate form (cute_index) gives Eq. 3's index for
    every element, and it is where the CuTe stride view (realised by numpy's
    as_strided over a packed buffer) finds B[k, n]."""
    k, n = np.meshgrid(np.arange(K), np.arange(N), indexing="ij")
    idx = L.cute_index(k, n, K, N, G)
    assert np.array_equal(idx, L.eq3_index(k, n, K, N, G))
    assert sorted(idx.ravel()) == list(range(K * N))          # a bijection onto the buffer
    rng = np.random.default_rng(K + N)
    B = rng.integers(0, 65535, size=(K, N), dtype=np.uint16)
    buf = L.pack(B, 1, G, P=2)
    assert np.array_equal(buf[idx], B)
    w = N // G
    view = np.lib.stride_tricks.as_strided(buf, shape=(K, G, w),
                                           strides=(w * buf.itemsize, K * w * buf.itemsize, buf.itemsize))
    assert np.array_equal(view[k, n // w, n % w], buf[idx])


def test_cute_index_worked_example():
    """The two-chiplet example of Sec. III-A: B[1, 5] with K = 4, N = 8 sits
    at CCL index 21 (chiplet 1's strip starts at 16)."""
    assert int(L.cute_index(1, 5, 4, 8, 2)) == 21


@pytest.mark.parametrize("R,Cc,Pr,Pc,P", [(64, 96, 2, 3, 4096), (256, 512, 2, 4, 65536),
                                          (48, 40, 4, 2, 256), (33, 17, 1, 1, 4096)])
def test_unpack_rows_is_a_row_slice_of_unpack(R, Cc, Pr, Pc, P):
    rng = np.random.default_rng(R * Cc)
    X = rng.integers(0, 65535, size=(R, Cc), dtype=np.uint16)
    buf = L.pack_reshape(X, Pr, Pc, P, fill=0xFFFF)
    for r0, r1 in ((0, R), (0, 1), (R // 3, R // 2 + 1), (R - 1, R), (5, 5)):
        assert np.array_equal(L.unpack_rows(buf, R, Cc, Pr, Pc, P, r0, r1), X[r0:r1])
    with pytest.raises(ValueError):
        L.unpack_rows(buf, R, Cc, Pr, Pc, P, 0, R + 1)


def test_two_chiplet_worked_example():
    """Sec. III-A: with two chiplets row-major alternates per-chiplet slices
    every 4 elements; CCL keeps 16 elements of one chiplet together."""
    g = GOLDEN["two_chiplet_example"]
    G, K, N = g["chiplets"], 4, 8
    # chiplet of each element, walked in memory order
    rowmajor_chip = [L.block_of(i // N, i % N, K, N, 1, G) for i in range(K * N)]
    r, c, valid = L.ccl_inverse(np.arange(K * N) * 2, K, N, 1, G, P=2)
    assert valid.all()
    ccl_chip = list(L.block_of(r, c, K, N, 1, G))
    assert set(_runs(rowmajor_chip)) == {g["rowmajor_run_elems"]}
    assert set(_runs(ccl_chip)) == {g["ccl_run_elems"]}
    # B[1, 5]: row-major index 13; Eq. 3: g = 1, n' = 1 -> 1*16 + 1*4 + 1 = 21
    assert L.eq2_index(1, 5, N) == 13
    assert int(L.ccl_offset(1, 5, K, N, 1, G, P=2)) // 2 == 21


def test_misalignment_slices():
    """Sec. II-B: row slices of 384 B, 2 KB, 7168 B (widths 768/4096/14336,
    4 chiplets, bf16); none is a whole number of pages."""
    g = GOLDEN["misalignment_slices"]
    for width, slice_bytes in zip(g["row_widths"], g["slice_bytes"]):
        rows = 3
        chips = [int(L.block_of(i // width, i % width, rows, width, 1, g["chiplets"]))
                 for i in range(rows * width)]
        runs = _runs(chips)
        assert set(runs) == {slice_bytes // g["elem_bytes"]}
        for P in g["page_sizes_checked"]:
            assert slice_bytes % P != 0


def test_fused_gate_up_slice_and_strip():
    g = GOLDEN["fused_gate_up_slice"]
    hr, wc = L.block_shape(2048, g["row_width"], 1, g["chiplets"])
    assert wc == g["slice_elems"]
    # a whole CCL strip of the Qwen3 gate/up weight (hidden 2048) is an exact
    # number of 4 KB pages, so CCL needs no padding there (Sec. III-B)
    strip = hr * wc * 2
    assert strip == 1572864 and strip % 4096 == 0
    assert L.strip_stride_bytes(2048, g["row_width"], 1, g["chiplets"], 4096) == strip


SHAPES = [(8, 16, 2, 2, 128), (12, 40, 3, 2, 256), (256, 512, 2, 4, 4096),
          (64, 96, 1, 8, 4096), (96, 64, 8, 1, 1024), (10, 10, 1, 1, 128), (384, 768, 4, 2, 65536)]


@pytest.mark.parametrize("R,Cc,Pr,Pc,P", SHAPES)
def test_map_is_bijection_with_inverse(R, Cc, Pr, Pc, P):
    r, c = np.meshgrid(np.arange(R), np.arange(Cc), indexing="ij")
    off = L.ccl_offset(r, c, R, Cc, Pr, Pc, P).reshape(-1)
    total = L.total_bytes(R, Cc, Pr, Pc, P)
    assert off.min() >= 0 and off.max() < total
    assert len(np.unique(off)) == R * Cc                    # injective
    r2, c2, valid = L.ccl_inverse(off, R, Cc, Pr, Pc, P)
    assert valid.all()
    assert np.array_equal(r2, r.reshape(-1)) and np.array_equal(c2, c.reshape(-1))
    # every element-aligned offset is either an element or padding
    all_off = np.arange(0, total, 2)
    _, _, v = L.ccl_inverse(all_off, R, Cc, Pr, Pc, P)
    assert int(v.sum()) == R * Cc


@pytest.mark.parametrize("R,Cc,Pr,Pc,P", SHAPES)
def test_each_strip_contiguous_and_page_aligned(R, Cc, Pr, Pc, P):
    """Sec. III-B: each chiplet's elements form one contiguous range whose
    start is page-aligned (the strip is padded to a page multiple)."""
    r, c = np.meshgrid(np.arange(R), np.arange(Cc), indexing="ij")
    off = L.ccl_offset(r, c, R, Cc, Pr, Pc, P)
    blk = L.block_of(r, c, R, Cc, Pr, Pc)
    hr, wc = R // Pr, Cc // Pc
    for b in range(Pr * Pc):
        o = np.sort(off[blk == b])
        assert o[0] % P == 0
        assert np.array_equal(o, o[0] + 2 * np.arange(hr * wc))


@pytest.mark.parametrize("R,Cc,Pr,Pc,P", SHAPES)
def test_pack_unpack_identity_and_reshape_form(R, Cc, Pr, Pc, P):
    rng = np.random.default_rng(R * 7 + Cc)
    X = rng.integers(0, 65535, size=(R, Cc), dtype=np.uint16)
    a = L.pack(X, Pr, Pc, P)
    b = L.pack_reshape(X, Pr, Pc, P)
    assert np.array_equal(a, b)
    assert np.array_equal(L.unpack(a, R, Cc, Pr, Pc, P), X)
    pad = L.padding_mask(R, Cc, Pr, Pc, P)
    assert int((~pad).sum()) == R * Cc
    assert np.all(a[pad] == 0)


def test_footprint_padding_ratios():
    """Padding only where a strip is not a page multiple: tiny 256x256 A on a
    2x2 grid has 32 KB strips -> 64x at 2 MB pages, 2x at 64 KB, 1x at 4 KB."""
    logical = 256 * 256 * 2
    assert L.total_bytes(256, 256, 2, 2, 4096) == logical
    assert L.total_bytes(256, 256, 2, 2, 65536) == 2 * logical
    assert L.total_bytes(256, 256, 2, 2, 2 * 1024 * 1024) == 64 * logical
    # Llama shapes need no padding at any page size
    for (R, Cc, Pr, Pc) in [(8192, 8192, 2, 4), (8192, 28672, 2, 4), (28672, 8192, 2, 4)]:
        for P in (4096, 65536, 2 * 1024 * 1024):
            assert L.total_bytes(R, Cc, Pr, Pc, P) == R * Cc * 2


def test_block_form_rejects_non_dividing_grid():
    with pytest.raises(ValueError):
        L.block_shape(10, 12, 3, 2)
