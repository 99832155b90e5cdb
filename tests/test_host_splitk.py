"""Host side of the split-K GEMM (ccl_gemm_splitk_workspace, ccl_gemm_splitk),
through the C ABI, with no GPU: the range count and workspace size, and
every argument check that runs before a device call.

The workspace holds one fp32 tile per (tile, K range); the tiles of all
partitions cover C exactly once, so its size is M * N * ranges * 4 bytes.
"""
import ctypes

import pytest

from paper_2606_11718_amd import ccl

BF16, FP8, FP32 = ccl.CCL_DT_BF16, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_FP32


def _ranges(ksteps: int, requested: int) -> int:
    """Non-empty ranges when ksteps are cut into ranges of ceil(ksteps / requested)."""
    per = -(-ksteps // requested)
    return -(-ksteps // per)


@pytest.mark.parametrize("M,N,K,G,Gr,ab", [
    (768, 2048, 4096, 8, 1, BF16),        # Qwen3 dW_down shape
    (2048, 1536, 4096, 8, 2, BF16),       # Qwen3 dW_gate/up shape
    (256, 512, 160, 1, 1, BF16),          # 5 K steps
    (256, 512, 320, 1, 1, FP8),           # 5 fp8 K steps of 64
    (1024, 1024, 16384, 8, 2, BF16),
    (8192, 28672, 8192, 8, 2, BF16),      # Llama-3.1-70B forward: already fills the chip
])
@pytest.mark.parametrize("requested", [1, 2, 3, 4, 7, 16])
def test_workspace_is_one_fp32_tile_per_tile_and_range(M, N, K, G, Gr, ab, requested):
    p = ccl.ccl_plan_typed(M, N, K, G, Gr, 4096, ab, BF16)
    ksteps = K // (64 if ab == FP8 else 32)
    got, nbytes = ccl.ccl_gemm_splitk_workspace(p, requested)
    assert got == _ranges(ksteps, requested)
    assert nbytes == (M * N * got * 4 if got > 1 else 0)


@pytest.mark.parametrize("M,N,K,G,Gr", [(768, 2048, 4096, 8, 1), (2048, 1536, 4096, 8, 2),
                                        (8192, 28672, 8192, 8, 2), (256, 512, 160, 1, 1),
                                        (256, 256, 8192, 1, 1), (1024, 768, 1024, 8, 8)])
def test_chosen_split_count_fills_an_xcd(M, N, K, G, Gr):
    """splits = 0: ranges = min(32 // tiles per XCD, K steps // 8, 16), at
    least 1, so that an XCD's 32 compute units get about one workgroup each
    and every range keeps at least 8 main-loop steps."""
    p = ccl.ccl_plan(M, N, K, G, Gr, 4096)
    _, _, wgs = ccl.ccl_debug_gemm_config(p)
    per_xcd = wgs // 8
    want = max(1, min(32 // per_xcd, (K // 32) // 8, 16))
    got, nbytes = ccl.ccl_gemm_splitk_workspace(p, 0)
    assert got == want
    assert nbytes == (M * N * got * 4 if got > 1 else 0)


def test_workspace_query_rejects_bad_arguments():
    lib = ccl.library()
    p = ccl.ccl_plan(768, 2048, 4096, 8, 1, 4096)
    s, n = ctypes.c_int(17), ctypes.c_int64(0)
    assert lib.ccl_gemm_splitk_workspace(p, ctypes.byref(s), ctypes.byref(n)) == 1
    s.value = -1
    assert lib.ccl_gemm_splitk_workspace(p, ctypes.byref(s), ctypes.byref(n)) == 1
    assert lib.ccl_gemm_splitk_workspace(p, None, ctypes.byref(n)) == 1
    assert lib.ccl_gemm_splitk_workspace(p, ctypes.byref(s), None) == 1
    assert lib.ccl_gemm_splitk_workspace(None, ctypes.byref(s), ctypes.byref(n)) == 1
    q = ccl.ccl_plan(384, 768, 384, 3, 1, 4096)              # 3 chiplets: no GEMM kernel
    s.value = 2
    assert lib.ccl_gemm_splitk_workspace(q, ctypes.byref(s), ctypes.byref(n)) == 3
    f = ccl.ccl_plan_typed(256, 512, 256, 4, 2, 4096, FP32, FP32)
    assert lib.ccl_gemm_splitk_workspace(f, ctypes.byref(s), ctypes.byref(n)) == 3


def test_splitk_gemm_argument_checks_before_any_device_call():
    lib = ccl.library()
    p = ccl.ccl_plan(768, 2048, 4096, 8, 1, 4096)
    _, need = ccl.ccl_gemm_splitk_workspace(p, 4)
    f = ctypes.c_float
    call = lambda s, ws, nb, a=4096: lib.ccl_gemm_splitk(p, f(1), a, 4096, f(0), 4096, s, ws, nb, None)
    assert call(0, 4096, need) == 1                 # the GEMM takes 1..16 ranges
    assert call(17, 4096, need) == 1
    assert call(4, None, need) == 1                 # no workspace
    assert call(4, 4096, need - 4) == 1             # workspace too small
    assert "workspace" in lib.ccl_last_error().decode()
    assert call(4, 4104, need) == 4                 # misaligned workspace
    assert call(4, 4096, need, a=4100) == 4         # misaligned operand
    assert lib.ccl_gemm_splitk(p, f(1), None, 4096, f(0), 4096, 4, 4096, need, None) == 1
    q = ccl.ccl_plan(384, 768, 384, 3, 1, 4096)
    assert lib.ccl_gemm_splitk(q, f(1), 4096, 4096, f(0), 4096, 2, 4096, 1 << 30, None) == 3


@pytest.mark.parametrize("splits", [1, 2, 4, 16])
def test_splitk_host_checks_pass_for_valid_calls(splits):
    """A valid call passes every host check and fails only at the device
    query on a host without a GPU; one range needs no workspace."""
    import torch
    if torch.cuda.device_count() > 0:      # placeholder pointers must never reach a device
        pytest.skip("needs a host without a GPU")
    lib = ccl.library()
    for ab, c in ((BF16, BF16), (BF16, FP32), (FP8, BF16)):
        p = ccl.ccl_plan_typed(768, 2048, 4096, 8, 1, 4096, ab, c)
        _, need = ccl.ccl_gemm_splitk_workspace(p, splits)
        ws = 4096 if need else None
        st = lib.ccl_gemm_splitk(p, ctypes.c_float(0.5), 4096, 4096, ctypes.c_float(1.0), 4096,
                                 splits, ws, need, None)
        msg = lib.ccl_last_error().decode()
        assert "internal" not in msg
        assert st == 5 and "hipGetDevice" in msg, msg


def test_noalloc_splitk_host_checks():
    """ccl_gemm_splitk_noalloc refuses, before any device call, workspaces
    beyond the library's static scratch, bad split counts and NULL operands;
    a request that fits gets as far as the device query."""
    import torch
    lib = ccl.library()
    big = ccl.ccl_plan(4096, 4096, 8192, 8, 2, 4096)
    splits, ws = ccl.ccl_gemm_splitk_workspace(big, 2)
    assert splits == 2 and ws == 4096 * 4096 * 2 * 4 > ccl.CCL_SCRATCH_BYTES
    assert lib.ccl_gemm_splitk_noalloc(big, 1.0, 4096, 4096, 0.0, 4096, 2, None) == 1
    assert "static scratch" in lib.ccl_last_error().decode()
    small = ccl.ccl_plan(768, 2048, 4096, 8, 1, 4096)
    for bad in (0, 17):
        assert lib.ccl_gemm_splitk_noalloc(small, 1.0, 4096, 4096, 0.0, 4096, bad, None) == 1
    assert lib.ccl_gemm_splitk_noalloc(small, 1.0, None, 4096, 0.0, 4096, 2, None) == 1
    assert lib.ccl_gemm_splitk_noalloc(small, 1.0, 4100, 4096, 0.0, 4096, 2, None) == 4
    for splits in (1, 2, 8):                    # dW_down fits up to 10 ranges
        assert ccl.ccl_gemm_splitk_workspace(small, splits)[1] <= ccl.CCL_SCRATCH_BYTES
    assert ccl.ccl_gemm_splitk_workspace(small, 16)[1] > ccl.CCL_SCRATCH_BYTES
    assert lib.ccl_gemm_splitk_noalloc(small, 1.0, 4096, 4096, 0.0, 4096, 16, None) == 1
    if torch.cuda.device_count() == 0:          # placeholder pointers never reach a device
        assert lib.ccl_gemm_splitk_noalloc(small, 1.0, 4096, 4096, 0.0, 4096, 2, None) == 5
        assert "hipGetDevice" in lib.ccl_last_error().decode()


def test_gemm_timeline_host_checks():
    """ccl_debug_gemm_timeline refuses, before any device call, NULL
    arguments, a timeline shorter than workgroups * waves * 64 bytes,
    misaligned pointers and fp8 plans."""
    import torch
    lib = ccl.library()
    p = ccl.ccl_plan(768, 2048, 4096, 8, 1, 4096)
    _, _, wgs = ccl.ccl_debug_gemm_config(p)
    need = wgs * 8 * 64
    call = lambda tl, nb, a=4096: lib.ccl_debug_gemm_timeline(p, a, 4096, 4096, tl, nb, None)
    assert call(None, need) == 1
    assert call(4096, need - 1) == 1
    assert "timeline smaller" in lib.ccl_last_error().decode()
    assert call(4104, need) == 4
    assert call(4096, need, a=4100) == 4
    f8 = ccl.ccl_plan_typed(768, 2048, 4096, 8, 1, 4096, FP8, BF16)
    assert lib.ccl_debug_gemm_timeline(f8, 4096, 4096, 4096, 4096, need, None) == 3
    if torch.cuda.device_count() == 0:          # placeholder pointers never reach a device
        assert call(4096, need) == 5
        assert "hipGetDevice" in lib.ccl_last_error().decode()
