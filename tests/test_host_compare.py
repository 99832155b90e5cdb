"""The row-block comparison that the GPU tests use on Llama-sized products
(tests/helpers.py), exercised on the CPU with CCL buffers the oracle packs:
an exact product compares equal, a single planted error anywhere in C is
seen, and every element is visited."""
import numpy as np
import pytest

from oracle import gemm as OG
from oracle import layout as OL
from tests.helpers import compare_in_row_blocks


@pytest.mark.parametrize("M,N,Gr,Gc,P,block", [(96, 64, 2, 4, 4096, 40), (256, 384, 2, 2, 256, 1024),
                                              (64, 128, 1, 8, 65536, 7)])
def test_row_block_compare_sees_every_element(M, N, Gr, Gc, P, block):
    rng = np.random.default_rng(M + N)
    ref = rng.standard_normal((M, N)).astype(np.float32).astype(np.float64)
    bits = ref.astype(np.float32).view(np.uint32)
    good = OL.pack_reshape(bits, Gr, Gc, P, fill=0x7FC00000)      # NaN in padding
    bad = good.copy()
    r, c = M - 1, N // 3
    off = int(OL.ccl_offset(r, c, M, N, Gr, Gc, P, 4)) // 4
    bad[off] = np.float32(ref[r, c] + 10.0).view(np.uint32)
    dec = lambda b: b.view(np.float32).astype(np.float64)
    errs = compare_in_row_blocks({"good": (good, Gr, Gc), "bad": (bad, Gr, Gc)}, M, N, P,
                                 lambda r0, r1: ref[r0:r1], dec, rows_per_block=block)
    assert errs["good"] == {"rel_fro": 0.0, "max_abs": 0.0, "max_ref": float(np.abs(ref).max())}
    assert errs["bad"]["max_abs"] == pytest.approx(10.0, rel=1e-6)
    assert not OG.within_tolerance(errs["bad"])
