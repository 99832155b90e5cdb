"""fp64 GEMM oracle and error metrics, Sec. II-B (C = A B).

The GEMM itself is unchanged by CCL (Sec. III-C): only operand addresses
change. The oracle therefore is the plain definition C[m, n] = sum_k A[m, k]
B[k, n], evaluated in float64 on the exact bf16 input values.

Precision: the paper evaluates BF16 GEMMs (Sec. IV-A). Reading: bf16
operands, fp32 accumulation, bf16 output rounded to nearest even; the order
of accumulation is free, so the GPU result is compared under a tolerance
(relative Frobenius error <= 5e-3 and max abs error <= 1e-2 * max|C_ref|).
Fig. 7 also sweeps the data type: fp8 (E4M3) operands and an fp32 output
are decoded exactly here and compared the same way.

Pinned by: integer (ternary) inputs against exact integer matmul, B = I,
and per-element math.fsum on random inputs (tests).
"""
from __future__ import annotations

import numpy as np


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def decode_fp8_e4m3(bits: np.ndarray) -> np.ndarray:
    """fp8 E4M3 bit patterns (uint8, the OCP 8-bit format with 4 exponent
    bits, bias 7, 3 mantissa bits, no infinities) -> exact float64 values.

    Exponent field 0 is subnormal: mantissa * 2^-9. S.1111.111 is NaN; every
    other pattern, including exponent 15, is finite (largest 448).
    """
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    ex = (b >> 3) & 0xF
    man = b & 0x7
    val = np.where(ex == 0, man * 2.0 ** -9, (1.0 + man / 8.0) * np.exp2(ex - 7.0))
    val = np.where((ex == 15) & (man == 7), np.nan, val)
    return sign * val


def decode(bits: np.ndarray) -> np.ndarray:
    """Exact float64 values of bf16 (uint16) or fp8 E4M3 (uint8) bit arrays;
    float arrays pass through."""
    if bits.dtype == np.uint16:
        return decode_bf16(bits)
    if bits.dtype == np.uint8:
        return decode_fp8_e4m3(bits)
    return np.asarray(bits, dtype=np.float64)


def gemm_fp64(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """C = A B in float64. A, B are float64, bf16 bits (uint16) or fp8 E4M3
    bits (uint8)."""
    A = decode(A)
    B = decode(B)
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
    return alpha * P + beta * decode(C)


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


class ErrorAccumulator:
    """errors() of a matrix that arrives in row blocks.

    The definition's sums of squares (of C_test - C_ref and of C_ref) and
    its two maxima are accumulated block by block in float64, so a product
    too large to hold twice on the host is still compared element by
    element. result() has the keys of errors().
    """

    def __init__(self):
        self.sq_diff = 0.0
        self.sq_ref = 0.0
        self.max_abs = 0.0
        self.max_ref = 0.0
        self.count = 0

    def add(self, C_test: np.ndarray, C_ref: np.ndarray) -> None:
        C_test = np.asarray(C_test, dtype=np.float64)
        C_ref = np.asarray(C_ref, dtype=np.float64)
        if C_test.shape != C_ref.shape:
            raise ValueError("block shapes differ")
        if C_ref.size == 0:
            return
        d = (C_test - C_ref).ravel()
        r = C_ref.ravel()
        self.sq_diff += float(np.dot(d, d))
        self.sq_ref += float(np.dot(r, r))
        self.max_abs = max(self.max_abs, float(np.max(np.abs(d))))
        self.max_ref = max(self.max_ref, float(np.max(np.abs(r))))
        self.count += C_ref.size

    def result(self) -> dict:
        d, r = self.sq_diff ** 0.5, self.sq_ref ** 0.5
        return {"rel_fro": d / r if r > 0 else d, "max_abs": self.max_abs,
                "max_ref": self.max_ref}


def within_tolerance(err: dict, rel_fro_tol: float = 5e-3, max_abs_frac: float = 1e-2) -> bool:
    return err["rel_fro"] <= rel_fro_tol and err["max_abs"] <= max_abs_frac * err["max_ref"]
