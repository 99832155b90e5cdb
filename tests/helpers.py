"""Shared helpers of the GPU tests (device transfers of bf16 bit arrays)."""
import numpy as np

CANARY = 0x7E1D          # bf16 bits written into padding / untouched areas


def torch_mod():
    import torch
    return torch


def to_dev(bits: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")


def from_dev(t) -> np.ndarray:
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy().view(np.uint16)


def dev_full(n_elems: int, value: int = CANARY):
    torch = torch_mod()
    v = value - 65536 if value >= 32768 else value
    return torch.full((n_elems,), v, dtype=torch.int16, device="cuda")


def with_ld(X: np.ndarray, ld: int, fill: int = CANARY) -> np.ndarray:
    """Copy of X (rows x cols) inside a wider rows x ld array."""
    out = np.full((X.shape[0], ld), fill, dtype=np.uint16)
    out[:, :X.shape[1]] = X
    return out
