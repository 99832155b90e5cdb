"""ctypes binding of libccl.so: the calls of include/ccl.h under the same names.

Argument marshalling only: every step runs in the HIP library. Device
buffers may be given as torch tensors (their data_ptr() is passed) or as
integer device addresses; `stream` may be a torch.cuda.Stream, an integer
hipStream_t, or None (torch's current stream when torch has initialised the
GPU, else the null stream). Errors raise CCLError with the library's status
and message. If libccl.so is not built, loading raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libccl.so")

CCL_A, CCL_B, CCL_C = 0, 1, 2
CCL_PLACE_RR, CCL_PLACE_COARSE, CCL_PLACE_CCL = 0, 1, 2
CCL_SCRATCH_BYTES = 64 << 20        # static split-K workspace of ccl_gemm_splitk_noalloc, per GPU
MAX_CHIPLETS = 64

STATUS_NAMES = {0: "CCL_OK", 1: "CCL_ERR_INVALID_ARG", 2: "CCL_ERR_UNALIGNED_PARTITION",
                3: "CCL_ERR_UNSUPPORTED", 4: "CCL_ERR_MISALIGNED_POINTER", 5: "CCL_ERR_HIP"}

# every symbol include/ccl.h declares
EXPORTED = ("ccl_plan", "ccl_plan_typed", "ccl_plan_destroy", "ccl_plan_grid", "ccl_plan_layout",
            "ccl_pack", "ccl_unpack", "ccl_gemm", "ccl_gemm_scaled", "ccl_gemm_splitk_workspace",
            "ccl_gemm_splitk", "ccl_gemm_splitk_noalloc", "ccl_gemm_rowmajor", "ccl_remote_bytes", "ccl_remote_bytes_l2", "ccl_status_string", "ccl_last_error",
            "ccl_debug_tile_of_wg", "ccl_debug_gemm_config", "ccl_debug_dispatch",
            "ccl_debug_gemm_timeline")


class CCLError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.status_name = STATUS_NAMES.get(status, str(status))
        super().__init__(f"{self.status_name}: {message}")


class _Layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("rows", "cols", "grid_r", "grid_c", "block_rows",
                                               "block_cols", "strip_bytes", "strip_stride_bytes",
                                               "total_bytes", "elem_bytes")]


class _Traffic(ctypes.Structure):
    _fields_ = [("accessed", ctypes.c_uint64 * 3), ("remote", ctypes.c_uint64 * 3),
                ("floor_bytes", ctypes.c_uint64), ("footprint", ctypes.c_uint64 * 3),
                ("remote_per_chiplet", ctypes.c_uint64 * MAX_CHIPLETS), ("chiplets", ctypes.c_int32)]


class _L2Config(ctypes.Structure):
    _fields_ = [("l2_bytes", ctypes.c_int64), ("ways", ctypes.c_int32), ("line_bytes", ctypes.c_int32),
                ("slots", ctypes.c_int32), ("k_step", ctypes.c_int32), ("traversal", ctypes.c_int32),
                ("threads", ctypes.c_int32), ("group_rows", ctypes.c_int32)]


class _L2Traffic(ctypes.Structure):
    _fields_ = [("accesses", ctypes.c_uint64 * 2), ("misses", ctypes.c_uint64 * 2),
                ("remote", ctypes.c_uint64 * 3),
                ("remote_per_chiplet", ctypes.c_uint64 * MAX_CHIPLETS), ("chiplets", ctypes.c_int32)]


_lib = None


def library() -> ctypes.CDLL:
    """Load libccl.so once (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run __graft_entry__.build() "
                          "or python -m paper_2606_11718_amd.build")
    # libccl.so needs libamdhip64.so.7. torch ships its own copy of the HIP
    # runtime under that soname; loading torch first makes the dynamic loader
    # hand libccl.so that same runtime, so one HIP runtime serves both (two
    # runtimes in one process do not share devices, memory or streams).
    import torch  # noqa: F401
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    sig = {
        "ccl_plan": [i64, i64, i64, i32, i32, i64, ctypes.POINTER(vp)],
        "ccl_plan_typed": [i64, i64, i64, i32, i32, i64, i32, i32, ctypes.POINTER(vp)],
        "ccl_plan_destroy": [vp],
        "ccl_plan_grid": [vp, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "ccl_plan_layout": [vp, i32, ctypes.POINTER(_Layout)],
        "ccl_pack": [vp, i32, vp, i64, i32, vp, vp],
        "ccl_unpack": [vp, i32, vp, vp, i64, vp],
        "ccl_gemm": [vp, vp, vp, vp, vp],
        "ccl_gemm_scaled": [vp, ctypes.c_float, vp, vp, ctypes.c_float, vp, vp],
        "ccl_gemm_splitk_workspace": [vp, ctypes.POINTER(i32), ctypes.POINTER(i64)],
        "ccl_gemm_splitk": [vp, ctypes.c_float, vp, vp, ctypes.c_float, vp, i32, vp, i64, vp],
        "ccl_gemm_splitk_noalloc": [vp, ctypes.c_float, vp, vp, ctypes.c_float, vp, i32, vp],
        "ccl_gemm_rowmajor": [vp, vp, vp, vp, i32, vp],
        "ccl_remote_bytes": [vp, i32, i32, ctypes.POINTER(_Traffic)],
        "ccl_remote_bytes_l2": [vp, i32, i32, ctypes.POINTER(_L2Config), ctypes.POINTER(_L2Traffic)],
        "ccl_debug_tile_of_wg": [vp, i64, ctypes.POINTER(i32), ctypes.POINTER(i64), ctypes.POINTER(i64)],
        "ccl_debug_gemm_config": [vp, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i64)],
        "ccl_debug_dispatch": [vp, vp, vp],
        "ccl_debug_gemm_timeline": [vp, vp, vp, vp, vp, i64, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.ccl_status_string.argtypes = [ctypes.c_int]
    lib.ccl_status_string.restype = ctypes.c_char_p
    lib.ccl_last_error.argtypes = []
    lib.ccl_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        raise CCLError(status, library().ccl_last_error().decode())


def _ptr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> int:
    if s is None:
        import sys
        torch = sys.modules.get("torch")
        if torch is not None and torch.cuda.is_initialized():
            return int(torch.cuda.current_stream().cuda_stream)
        return 0
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


class Plan:
    """Owns a ccl_plan_t; destroyed with the object."""

    def __init__(self, handle: int, args: tuple):
        self.handle = handle
        self.args = args

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.ccl_plan_destroy(self.handle)
            self.handle = None

    @property
    def _as_parameter_(self):
        return ctypes.c_void_p(self.handle)


@dataclass
class Layout:
    rows: int
    cols: int
    grid_r: int
    grid_c: int
    block_rows: int
    block_cols: int
    strip_bytes: int
    strip_stride_bytes: int
    total_bytes: int
    elem_bytes: int


CCL_DT_BF16, CCL_DT_FP8_E4M3, CCL_DT_FP32 = 0, 1, 2


def ccl_plan(M: int, N: int, K: int, chiplets: int, grid_rows: int, page_bytes: int) -> Plan:
    h = ctypes.c_void_p()
    _check(library().ccl_plan(M, N, K, chiplets, grid_rows, page_bytes, ctypes.byref(h)))
    return Plan(h.value, (M, N, K, chiplets, grid_rows, page_bytes))


def ccl_plan_typed(M: int, N: int, K: int, chiplets: int, grid_rows: int, page_bytes: int,
                   ab_type: int, c_type: int) -> Plan:
    h = ctypes.c_void_p()
    _check(library().ccl_plan_typed(M, N, K, chiplets, grid_rows, page_bytes, ab_type, c_type,
                                    ctypes.byref(h)))
    return Plan(h.value, (M, N, K, chiplets, grid_rows, page_bytes, ab_type, c_type))


def ccl_plan_grid(plan: Plan) -> tuple[int, int]:
    r, c = ctypes.c_int(), ctypes.c_int()
    _check(library().ccl_plan_grid(plan, ctypes.byref(r), ctypes.byref(c)))
    return r.value, c.value


def ccl_plan_layout(plan: Plan, op: int) -> Layout:
    out = _Layout()
    _check(library().ccl_plan_layout(plan, op, ctypes.byref(out)))
    return Layout(*(getattr(out, f) for f, _ in _Layout._fields_))


def ccl_pack(plan: Plan, op: int, src, ld: int, src_trans: int, dst_ccl, stream=None) -> None:
    _check(library().ccl_pack(plan, op, _ptr(src), ld, src_trans, _ptr(dst_ccl), _stream(stream)))


def ccl_unpack(plan: Plan, op: int, src_ccl, dst, ld: int, stream=None) -> None:
    _check(library().ccl_unpack(plan, op, _ptr(src_ccl), _ptr(dst), ld, _stream(stream)))


def ccl_gemm(plan: Plan, A_ccl, B_ccl, C_ccl, stream=None) -> None:
    _check(library().ccl_gemm(plan, _ptr(A_ccl), _ptr(B_ccl), _ptr(C_ccl), _stream(stream)))


def ccl_gemm_scaled(plan: Plan, alpha: float, A_ccl, B_ccl, beta: float, C_ccl, stream=None) -> None:
    _check(library().ccl_gemm_scaled(plan, alpha, _ptr(A_ccl), _ptr(B_ccl), beta, _ptr(C_ccl),
                                     _stream(stream)))


def ccl_gemm_splitk_workspace(plan: Plan, splits: int = 0) -> tuple[int, int]:
    """(K ranges used, workspace bytes) for a requested split count (0: choose)."""
    s = ctypes.c_int(splits)
    nbytes = ctypes.c_int64(0)
    _check(library().ccl_gemm_splitk_workspace(plan, ctypes.byref(s), ctypes.byref(nbytes)))
    return s.value, nbytes.value


def ccl_gemm_splitk(plan: Plan, alpha: float, A_ccl, B_ccl, beta: float, C_ccl, splits: int,
                    workspace, workspace_bytes: int, stream=None) -> None:
    _check(library().ccl_gemm_splitk(plan, alpha, _ptr(A_ccl), _ptr(B_ccl), beta, _ptr(C_ccl),
                                     splits, _ptr(workspace), workspace_bytes, _stream(stream)))


def ccl_gemm_splitk_noalloc(plan: Plan, alpha: float, A_ccl, B_ccl, beta: float, C_ccl,
                            splits: int, stream=None) -> None:
    _check(library().ccl_gemm_splitk_noalloc(plan, ctypes.c_float(alpha), _ptr(A_ccl),
                                             _ptr(B_ccl), ctypes.c_float(beta), _ptr(C_ccl),
                                             splits, _stream(stream)))


def ccl_gemm_rowmajor(plan: Plan, A, B, C, remap: int, stream=None) -> None:
    _check(library().ccl_gemm_rowmajor(plan, _ptr(A), _ptr(B), _ptr(C), remap, _stream(stream)))


CCL_TRAFFIC_A_TRANS, CCL_TRAFFIC_B_TRANS, CCL_TRAFFIC_C_READ = 1, 2, 4


def ccl_remote_bytes(plan: Plan, placement: int, flags: int) -> dict:
    t = _Traffic()
    _check(library().ccl_remote_bytes(plan, placement, flags, ctypes.byref(t)))
    return {
        "accessed": list(t.accessed),
        "remote": list(t.remote),
        "remote_per_chiplet": list(t.remote_per_chiplet[:t.chiplets]),
        "floor": int(t.floor_bytes),
        "footprint": list(t.footprint),
    }


def ccl_remote_bytes_l2(plan: Plan, placement: int, flags: int, *, l2_bytes: int,
                        slots: int, ways: int = 16, line_bytes: int = 128, k_step: int = 64,
                        traversal: int = 0, threads: int = 0, group_rows: int = 0) -> dict:
    cfg = _L2Config(l2_bytes, ways, line_bytes, slots, k_step, traversal, threads, group_rows)
    t = _L2Traffic()
    _check(library().ccl_remote_bytes_l2(plan, placement, flags, ctypes.byref(cfg),
                                         ctypes.byref(t)))
    return {
        "accesses": list(t.accesses),
        "misses": list(t.misses),
        "remote": list(t.remote),
        "remote_per_chiplet": list(t.remote_per_chiplet[:t.chiplets]),
    }


def ccl_status_string(status: int) -> str:
    return library().ccl_status_string(status).decode()


def ccl_last_error() -> str:
    return library().ccl_last_error().decode()


def ccl_debug_tile_of_wg(plan: Plan, wg: int) -> tuple[int, int, int]:
    x, tm, tn = ctypes.c_int(), ctypes.c_int64(), ctypes.c_int64()
    _check(library().ccl_debug_tile_of_wg(plan, wg, ctypes.byref(x), ctypes.byref(tm), ctypes.byref(tn)))
    return x.value, tm.value, tn.value


def ccl_debug_gemm_config(plan: Plan) -> tuple[int, int, int]:
    r, c, w = ctypes.c_int(), ctypes.c_int(), ctypes.c_int64()
    _check(library().ccl_debug_gemm_config(plan, ctypes.byref(r), ctypes.byref(c), ctypes.byref(w)))
    return r.value, c.value, w.value


def ccl_debug_dispatch(plan: Plan, out, stream=None) -> None:
    _check(library().ccl_debug_dispatch(plan, _ptr(out), _stream(stream)))


def ccl_debug_gemm_timeline(plan: Plan, A_ccl, B_ccl, C_ccl, timeline, timeline_bytes: int,
                            stream=None) -> None:
    _check(library().ccl_debug_gemm_timeline(plan, _ptr(A_ccl), _ptr(B_ccl), _ptr(C_ccl),
                                             _ptr(timeline), timeline_bytes, _stream(stream)))
