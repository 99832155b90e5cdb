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


def compare_in_row_blocks(outputs: dict, M: int, N: int, P: int, ref_rows, decode_c,
                          rows_per_block: int = 1024) -> dict:
    """Element-by-element comparison of whole GPU products with the fp64
    oracle, for products too large to hold twice in fp64 on the host.

    outputs maps a key to (CCL buffer of C copied to the host, Gr, Gc);
    ref_rows(r0, r1) returns the oracle's fp64 rows r0 .. r1-1 of C, computed
    once per block and shared by every output. decode_c turns the unpacked
    bits of C into float64. Returns {key: errors dict over all of C}.
    """
    from oracle import gemm as OG
    from oracle import layout as OL
    accs = {k: OG.ErrorAccumulator() for k in outputs}
    for r0 in range(0, M, rows_per_block):
        r1 = min(M, r0 + rows_per_block)
        ref = ref_rows(r0, r1)
        for key, (buf, gr, gc) in outputs.items():
            accs[key].add(decode_c(OL.unpack_rows(buf, M, N, gr, gc, P, r0, r1)), ref)
    for key, acc in accs.items():
        assert acc.count == M * N, (key, acc.count)
    return {k: a.result() for k, a in accs.items()}
