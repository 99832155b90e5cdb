"""GEMM on Chiplet-Contiguous Layout operands for MI355X (gfx950).

The work is done by libccl.so (HIP kernels + host plan, C ABI in
include/ccl.h); `ccl` is its ctypes binding with the same names.
"""
from . import ccl  # noqa: F401
from .ccl import (CCL_A, CCL_B, CCL_C, CCL_PLACE_RR, CCL_PLACE_COARSE, CCL_PLACE_CCL,  # noqa: F401
                  CCL_TRAFFIC_A_TRANS, CCL_TRAFFIC_B_TRANS, CCL_TRAFFIC_C_READ,
                  CCL_DT_BF16, CCL_DT_FP8_E4M3, CCL_DT_FP32,
                  CCLError, ccl_plan, ccl_plan_typed, ccl_plan_grid, ccl_plan_layout, ccl_pack, ccl_unpack,
                  ccl_gemm, ccl_gemm_scaled, ccl_gemm_splitk_workspace, ccl_gemm_splitk,
                  ccl_gemm_rowmajor, ccl_remote_bytes, ccl_remote_bytes_l2, ccl_status_string,
                  ccl_last_error)
