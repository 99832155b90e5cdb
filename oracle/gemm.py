"""fp64 GEMM oracle and error metrics, Sec. II-B (C = A B).

The GEMM itself is unchanged by CCL (Sec. III-C): only operand addresses
change. The oracle therefore is the plain definition C[m, n] = sum_k A[m, k]
B[k, n], evaluated in float64 on the exact bf16 input values.

Precision: the paper evaluates BF16 GEMMs (Sec. IV-A). Reading: bf16
operands, fp32 accumulation, bf16 output rounded to nearest even; the order
of accumulation is free, so the GPU result is compared under a tolerance
(relative Frobenius error <= 5e-3 and max abs error <= 1e-2 * max|C_ref|).

Pinned by: integer (ternary) inputs against exact integer matmul, B = I,
and per-element math.fsum on random inputs (tests).
"""
from __future__ import annotations

import numpy as np


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def gemm_fp64(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """C = A B in float64. A, B are float64 (or bf16 bits as uint16)."""
    if A.dtype == np.uint16:
        A = decode_bf16(A)
    if B.dtype == np.uint16:
        B = decode_bf16(B)
    if A.shape[1] != B.shape[0]:
        raise ValueError("inner dimensions differ")
    return A @ B


def gemm_scaled_fp64(A, B, C, alpha: float, beta: float) -> np.ndarray:
    """alpha A B + beta C in float64 (the BLAS form of Sec. II-B).

    As in BLAS, beta == 0 means C is not read at all (its values, NaN
    included, do not matter).
    """
    P = gemm_fp64(A, B)
    if beta == 0:
        return alpha * P
    if C.dtype == np.uint16:
        C = decode_bf16(C)
    return alpha * P + beta * C


def gemm_entries(A: np.ndarray, B: np.ndarray, rows: np.ndarray, cols: np.ndarray) -> np.ndarray:
    """C[rows[i], cols[i]] for sampled output positions, in float64.

    A holds only the rows needed (indexed by rows), B is K x N (both may be
    bf16 bits). Used where the full product is too large for the host.
    """
    if A.dtype == np.uint16:
        A = decode_bf16(A)
    if B.dtype == np.uint16:
        B = decode_bf16(B)
    return np.einsum("ik,ki->i", A[rows], B[:, cols])


def errors(C_test: np.ndarray, C_ref: np.ndarray) -> dict:
    """rel_fro = ||C_test - C_ref||_F / ||C_ref||_F, max_abs, max_ref."""
    C_test = np.asarray(C_test, dtype=np.float64)
    C_ref = np.asarray(C_ref, dtype=np.float64)
    d = C_test - C_ref
    ref_norm = float(np.linalg.norm(C_ref))
    return {
        "rel_fro": float(np.linalg.norm(d)) / ref_norm if ref_norm > 0 else float(np.linalg.norm(d)),
        "max_abs": float(np.max(np.abs(d))) if d.size else 0.0,
        "max_ref": float(np.max(np.abs(C_ref))) if C_ref.size else 0.0,
    }


def within_tolerance(err: dict, rel_fro_tol: float = 5e-3, max_abs_frac: float = 1e-2) -> bool:
    return err["rel_fro"] <= rel_fro_tol and err["max_abs"] <= max_abs_frac * err["max_ref"]
