"""The Chiplet-Contiguous Layout (CCL) address map, Sec. III-B, Eq. 1-3.

Paper form (B of K x N split along N over G chiplets, Eq. 1-3):
    w = N / G,  g = floor(n / w),  n' = n mod w
    index_row(k, n) = k * N + n                      (Eq. 2)
    index_CCL(k, n) = g * K * w + k * w + n'         (Eq. 3)
so chiplet g's data is one contiguous strip of K*w elements. Sec. III-C gives
the same map as a CuTe-style view: shape (K, G, N/G) with strides (w, K*w, 1).

Block form used for every operand (reading: Sec. III-C applies CCL to A, B
and C; a 2-D grid is the natural extension of Eq. 3). An R x Cc operand with
a (Pr, Pc) block grid has blocks of hr = R/Pr rows and wc = Cc/Pc columns:
    b(r, c)   = floor(r / hr) * Pc + floor(c / wc)          (block = chiplet)
    off(r, c) = b * S + ((r mod hr) * wc + (c mod wc)) * e   (bytes)
where S = ceil(hr * wc * e / P) * P pads each strip to a whole number of
pages (Sec. III-B: the full chiplet-local strip is aligned to the page
boundary). With Pr = 1, Pc = G and no padding, off/e is exactly Eq. 3.
Padding bytes belong to no element.

Pinned by: Eq. 3 and the CuTe stride form (two independent formulas), the
two-chiplet worked example of Sec. III-A, the slice arithmetic of Sec. II-B,
bijection / contiguity / alignment properties, and pack == numpy reshape.
"""
from __future__ import annotations

import numpy as np


def block_shape(R: int, Cc: int, Pr: int, Pc: int) -> tuple[int, int]:
    if R % Pr or Cc % Pc:
        raise ValueError("grid does not divide the operand")
    return R // Pr, Cc // Pc


def strip_stride_bytes(R: int, Cc: int, Pr: int, Pc: int, P: int, e: int = 2) -> int:
    """Bytes from the start of one strip to the next (strip padded to P)."""
    hr, wc = block_shape(R, Cc, Pr, Pc)
    return -(-(hr * wc * e) // P) * P


def total_bytes(R: int, Cc: int, Pr: int, Pc: int, P: int, e: int = 2) -> int:
    return Pr * Pc * strip_stride_bytes(R, Cc, Pr, Pc, P, e)


# --- Sec. III-B, Eq. 1-3 as printed (B split along N only) -------------------

def eq1(n, w):
    """Eq. 1: chiplet index g and intra-chiplet column n'."""
    return n // w, n % w


def eq2_index(k, n, N):
    """Eq. 2: row-major element index."""
    return k * N + n


def eq3_index(k, n, K, N, G):
    """Eq. 3: CCL element index of B[k, n], B split along N over G chiplets."""
    w = N // G
    g, n_ = eq1(n, w)
    return g * K * w + k * w + n_


def cute_index(k, n, K, N, G):
    """Sec. III-C view: coordinate (k, g, n') under strides (w, K*w, 1)."""
    w = N // G
    g, n_ = n // w, n - (n // w) * w
    return k * w + g * (K * w) + n_ * 1


# --- block form over any operand -----------------------------------------------

def block_of(r, c, R, Cc, Pr, Pc):
    hr, wc = block_shape(R, Cc, Pr, Pc)
    return (np.asarray(r) // hr) * Pc + (np.asarray(c) // wc)


def ccl_offset(r, c, R, Cc, Pr, Pc, P, e=2):
    """Byte offset of logical element (r, c) in the CCL buffer."""
    hr, wc = block_shape(R, Cc, Pr, Pc)
    S = strip_stride_bytes(R, Cc, Pr, Pc, P, e)
    r = np.asarray(r, dtype=np.int64)
    c = np.asarray(c, dtype=np.int64)
    b = (r // hr) * Pc + (c // wc)
    return b * S + ((r % hr) * wc + (c % wc)) * e


def ccl_inverse(off, R, Cc, Pr, Pc, P, e=2):
    """Inverse map: byte offset -> (r, c, valid). valid is False on padding."""
    hr, wc = block_shape(R, Cc, Pr, Pc)
    S = strip_stride_bytes(R, Cc, Pr, Pc, P, e)
    off = np.asarray(off, dtype=np.int64)
    b = off // S
    q = (off % S) // e
    valid = (q < hr * wc) & (off % e == 0) & (b < Pr * Pc) & (off >= 0)
    qv = np.where(valid, q, 0)
    r = (b // Pc) * hr + qv // wc
    c = (b % Pc) * wc + qv % wc
    return r, c, valid


def pack(X: np.ndarray, Pr: int, Pc: int, P: int, fill: int = 0) -> np.ndarray:
    """Row-major R x Cc array -> CCL buffer (scatter through ccl_offset).

    Padding elements hold `fill`. Element type is kept (bf16 bits: uint16).
    """
    R, Cc = X.shape
    e = X.dtype.itemsize
    out = np.full(total_bytes(R, Cc, Pr, Pc, P, e) // e, fill, dtype=X.dtype)
    r, c = np.meshgrid(np.arange(R), np.arange(Cc), indexing="ij")
    out[ccl_offset(r, c, R, Cc, Pr, Pc, P, e) // e] = X
    return out


def pack_reshape(X: np.ndarray, Pr: int, Pc: int, P: int, fill: int = 0) -> np.ndarray:
    """Same result as pack(), built as a reshape/transpose of the blocks.

    (R, Cc) -> (Pr, hr, Pc, wc) -> (Pr, Pc, hr, wc): block-major, each block
    row-major; then each strip is padded to S bytes.
    """
    R, Cc = X.shape
    e = X.dtype.itemsize
    hr, wc = block_shape(R, Cc, Pr, Pc)
    S = strip_stride_bytes(R, Cc, Pr, Pc, P, e) // e
    strips = X.reshape(Pr, hr, Pc, wc).transpose(0, 2, 1, 3).reshape(Pr * Pc, hr * wc)
    out = np.full((Pr * Pc, S), fill, dtype=X.dtype)
    out[:, :hr * wc] = strips
    return out.reshape(-1)


def unpack(buf: np.ndarray, R: int, Cc: int, Pr: int, Pc: int, P: int) -> np.ndarray:
    """CCL buffer -> row-major R x Cc array (gather through ccl_offset)."""
    e = buf.dtype.itemsize
    r, c = np.meshgrid(np.arange(R), np.arange(Cc), indexing="ij")
    return buf[ccl_offset(r, c, R, Cc, Pr, Pc, P, e) // e]


def unpack_rows(buf: np.ndarray, R: int, Cc: int, Pr: int, Pc: int, P: int,
                r0: int, r1: int) -> np.ndarray:
    """Rows r0 .. r1-1 of the row-major operand held in a CCL buffer: the
    gather of unpack(), restricted to those rows."""
    if not 0 <= r0 <= r1 <= R:
        raise ValueError("row range outside the operand")
    e = buf.dtype.itemsize
    r, c = np.meshgrid(np.arange(r0, r1), np.arange(Cc), indexing="ij")
    return buf[ccl_offset(r, c, R, Cc, Pr, Pc, P, e) // e]


def padding_mask(R: int, Cc: int, Pr: int, Pc: int, P: int, e: int = 2) -> np.ndarray:
    """Boolean mask over the buffer's elements: True where padding."""
    n = total_bytes(R, Cc, Pr, Pc, P, e) // e
    _, _, valid = ccl_inverse(np.arange(n, dtype=np.int64) * e, R, Cc, Pr, Pc, P, e)
    return ~valid


def operand_shape(op: str, M: int, N: int, K: int) -> tuple[int, int]:
    return {"A": (M, K), "B": (K, N), "C": (M, N)}[op]
