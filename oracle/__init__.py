"""CPU oracle for GEMM on Chiplet-Contiguous Layout (CCL) operands.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import anything from here. The product path
(the HIP library and its Python binding) never imports, calls or links it.

Plain, slow, obviously correct numpy in float64 / int64:
  layout   the CCL address map (Sec. III-B, Eq. 1-3), its inverse, pack/unpack
  traffic  the integer remote-HBM-byte model under 4 KB round-robin
           interleave, coarse locality-aware placement and CCL (Sec. IV-A)
  l2sim    the remote-HBM traffic with a private set-associative LRU L2 per
           chiplet (Sec. IV-A simulation framework)
  gemm     the fp64 GEMM C = AB (Sec. II-B) and the error metrics
  plan     partition validity, tile ownership and automatic grid choice

Every reading of the paper made where it is silent or ambiguous is listed in
the module that uses it. Parity status of each function is stated in its
docstring ("pinned by ..." or "parity unpinned").
"""
from . import layout, traffic, l2sim, gemm, plan  # noqa: F401
