"""Seeded synthetic inputs for the CCL GEMM workloads.

This module only draws numbers and names shapes. It holds no layout, traffic
or GEMM arithmetic, so both the CPU oracle and the GPU path can take their
inputs from it without sharing any of the method's code.

Workloads (LLM FFN GEMMs, Sec. IV-A "Workloads"; bf16 operands):
  tiny        C[256x512] = A[256x256] B[256x512], U(-1,1), 4 chiplets, grid 2x2
  qwen_fwd    X[4096x2048] W_gate_up[2048x1536] (Qwen3-30B expert, fused gate+up)
  qwen_bwd    dW_down = H^T dY and dH = dY W_down^T (H 4096x768, dY 4096x2048)
  llama_fwd   X[8192x8192] W_up[8192x28672]; H[8192x28672] W_down[28672x8192]
  llama_bwd   dW_up = X^T dY and dX = dY W_up^T (dY 8192x28672)

The sweep of Sec. IV-A: the FFN gate/up and down projections of both models,
in the forward pass and both backward GEMMs (dX, dW), at 4K, 8K and 16K
tokens: 36 GEMM shapes (FFN_SWEEP; shapes only, no data).

Seeds: 1000 * workload number + index of the tensor in its workload, in
order of first appearance. Normal distributions are parameterised by their
standard deviation.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PAGE_4K = 4096
PAGE_64K = 65536
PAGE_2M = 2 * 1024 * 1024


@dataclass(frozen=True)
class Tensor:
    name: str
    rows: int
    cols: int
    dist: str          # "uniform" (U(-a,a)) or "normal" (N(0, a))
    scale: float       # a
    seed: int


@dataclass(frozen=True)
class Gemm:
    """One GEMM C = A B, A (M x K), B (K x N), as the GEMM sees them.

    a_src / b_src name the stored tensor; a_trans / b_trans say that the
    stored tensor is the transpose of the logical operand (e.g. H for H^T).
    grid_rows = 0 asks the plan to choose the grid itself.
    """
    name: str
    M: int
    N: int
    K: int
    a_src: str
    a_trans: int
    b_src: str
    b_trans: int
    chiplets: int
    grids: tuple          # tuple of grid_rows values to run (0 = automatic)
    pages: tuple          # page sizes in bytes

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K


@dataclass(frozen=True)
class Workload:
    number: int
    name: str
    tensors: dict = field(default_factory=dict)
    gemms: tuple = ()


def _t(number, idx, name, rows, cols, dist, scale):
    return Tensor(name, rows, cols, dist, scale, 1000 * number + idx)


def _workloads():
    w = {}
    n = 1
    w["tiny"] = Workload(n, "tiny", {
        "A": _t(n, 0, "A", 256, 256, "uniform", 1.0),
        "B": _t(n, 1, "B", 256, 512, "uniform", 1.0),
    }, (Gemm("tiny", 256, 512, 256, "A", 0, "B", 0, 4, (2,), (PAGE_4K,)),))
    n = 2
    w["qwen_fwd"] = Workload(n, "qwen_fwd", {
        "X": _t(n, 0, "X", 4096, 2048, "normal", 1.0),
        "W_gate_up": _t(n, 1, "W_gate_up", 2048, 1536, "normal", 0.02),
    }, (Gemm("qwen_gate_up", 4096, 1536, 2048, "X", 0, "W_gate_up", 0, 8, (2,), (PAGE_4K,)),))
    n = 3
    w["qwen_bwd"] = Workload(n, "qwen_bwd", {
        "H": _t(n, 0, "H", 4096, 768, "normal", 1.0),
        "dY": _t(n, 1, "dY", 4096, 2048, "normal", 1e-2),
        "W_down": _t(n, 2, "W_down", 768, 2048, "normal", 0.02),
    }, (Gemm("qwen_dW_down", 768, 2048, 4096, "H", 1, "dY", 0, 8, (0,), (PAGE_4K,)),
        Gemm("qwen_dH", 4096, 768, 2048, "dY", 0, "W_down", 1, 8, (0,), (PAGE_4K,))))
    n = 4
    w["llama_fwd"] = Workload(n, "llama_fwd", {
        "X": _t(n, 0, "X", 8192, 8192, "normal", 1.0),
        "W_up": _t(n, 1, "W_up", 8192, 28672, "normal", 0.02),
        "H": _t(n, 2, "H", 8192, 28672, "normal", 1.0),
        "W_down": _t(n, 3, "W_down", 28672, 8192, "normal", 0.02),
    }, (Gemm("llama_up", 8192, 28672, 8192, "X", 0, "W_up", 0, 8, (2,), (PAGE_4K,)),
        Gemm("llama_down", 8192, 8192, 28672, "H", 0, "W_down", 0, 8, (2,), (PAGE_4K,))))
    n = 5
    sweep_grids = (1, 2, 4, 8)
    sweep_pages = (PAGE_4K, PAGE_64K, PAGE_2M)
    w["llama_bwd"] = Workload(n, "llama_bwd", {
        "X": _t(n, 0, "X", 8192, 8192, "normal", 1.0),
        "dY": _t(n, 1, "dY", 8192, 28672, "normal", 1e-2),
        "W_up": _t(n, 2, "W_up", 8192, 28672, "normal", 0.02),
    }, (Gemm("llama_dW_up", 8192, 28672, 8192, "X", 1, "dY", 0, 8, sweep_grids, sweep_pages),
        Gemm("llama_dX", 8192, 8192, 28672, "dY", 0, "W_up", 1, 8, sweep_grids, sweep_pages)))
    return w


WORKLOADS = _workloads()


@dataclass(frozen=True)
class SweepGemm:
    """One GEMM of the FFN sweep: C = A B with A (M x K), B (K x N)."""
    model: str
    tokens: int
    proj: str            # "gate_up" or "down"
    pass_: str           # "fwd" (Y = X W), "dX" (dY W^T), "dW" (X^T dY)
    M: int
    N: int
    K: int
    a_trans: int         # A stored transposed (X^T held as X)
    b_trans: int         # B stored transposed (W^T held as W)

    @property
    def name(self) -> str:
        return f"{self.model}/{self.proj}/{self.pass_}/{self.tokens // 1024}K"


# hidden size, gate/up output width, down input width
FFN_MODELS = {
    "qwen3_30b": (2048, 1536, 768),        # one expert MLP, gate and up fused (2 x 768)
    "llama31_70b": (8192, 28672, 28672),   # the up (or gate) projection, as in llama_fwd
}
SWEEP_TOKENS = (4096, 8192, 16384)


def _ffn_sweep():
    out = []
    for model, (d, fg, f) in FFN_MODELS.items():
        for T in SWEEP_TOKENS:
            for proj, din, dout in (("gate_up", d, fg), ("down", f, d)):
                out.append(SweepGemm(model, T, proj, "fwd", T, dout, din, 0, 0))
                out.append(SweepGemm(model, T, proj, "dX", T, din, dout, 0, 1))
                out.append(SweepGemm(model, T, proj, "dW", din, dout, T, 1, 0))
    return tuple(out)


FFN_SWEEP = _ffn_sweep()


def gemm_by_name(name: str) -> tuple[Workload, Gemm]:
    for wl in WORKLOADS.values():
        for g in wl.gemms:
            if g.name == name:
                return wl, g
    raise KeyError(name)


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 bf16 bit patterns, round to nearest even.

    Inputs are finite draws, so no NaN/Inf handling is needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def round_to_fp8_e4m3_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> uint8 fp8 E4M3 (OCP) bit patterns, round to nearest
    even (torch's conversion). Draws stay far inside the +-448 range."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def draw_array_fp8(seed: int, rows: int, cols: int, dist: str = "normal", scale: float = 1.0) -> np.ndarray:
    """Draw an ad-hoc (rows x cols) fp8 E4M3 bit array: the same float32 draw
    as draw_array, rounded to fp8 instead of bf16."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = rows * cols
    if dist == "uniform":
        x = rng.uniform(-scale, scale, size=n).astype(np.float32)
    elif dist == "normal":
        x = rng.standard_normal(size=n, dtype=np.float32) * np.float32(scale)
    elif dist == "ternary":
        x = rng.integers(-1, 2, size=n).astype(np.float32)
    else:
        raise ValueError(dist)
    return round_to_fp8_e4m3_bits(x).reshape(rows, cols)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def draw(t: Tensor, rows: slice | None = None) -> np.ndarray:
    """Draw tensor t as a (rows x cols) uint16 array of bf16 bits.

    The draw is PCG64(seed) in float32, row-major, then rounded to bf16, so
    any row range can be regenerated without the rest (`rows` selects it;
    the stream is consumed in row-major order, so a row range costs the
    draws before it as well).
    """
    rng = np.random.Generator(np.random.PCG64(t.seed))
    n = t.rows * t.cols
    if t.dist == "uniform":
        x = rng.uniform(-t.scale, t.scale, size=n).astype(np.float32)
    elif t.dist == "normal":
        x = rng.standard_normal(size=n, dtype=np.float32) * np.float32(t.scale)
    elif t.dist == "ternary":
        x = rng.integers(-1, 2, size=n).astype(np.float32)
    else:
        raise ValueError(t.dist)
    out = round_to_bf16_bits(x).reshape(t.rows, t.cols)
    if rows is not None:
        out = np.ascontiguousarray(out[rows])
    return out


def draw_array(seed: int, rows: int, cols: int, dist: str = "normal", scale: float = 1.0) -> np.ndarray:
    """Draw an ad-hoc (rows x cols) bf16-bit array (edge-case tests)."""
    return draw(Tensor("adhoc", rows, cols, dist, scale, seed))
