"""Remote-HBM traffic of the FFN GEMM sweep under each placement (Sec. IV-A).

For every GEMM of workloads.FFN_SWEEP (Qwen3-30B and Llama-3.1-70B FFN
gate/up and down projections; forward, dX, dW; 4K/8K/16K tokens) and every
placement:
  * RR at 4 KB, 64 KB and 2 MB pages (fixed-granularity interleave),
  * COARSE (G contiguous page-granular chunks per tensor, Coarse LA),
  * CCL (strips padded to 4 KB pages),
the remote bytes are minimised over the tile-aligned output-partition grids
and the two tile traversal orders, as the paper reports each placement in
its best configuration. Two traffic models are available, both computed by
libccl.so: "l2" (ccl_remote_bytes_l2, a private LRU L2 per chiplet) and
"charge" (ccl_remote_bytes: no cache, every tile's panels charged).

A GEMM is coarse-optimal when COARSE reaches CCL's traffic (splitting every
operand into G contiguous blocks is already locality-optimal) and
fine-optimal otherwise. Ratios are summarised by geometric means (Sec. IV-A
metrics).

    python -m paper_2606_11718_amd.sweep --setting mi300x_like --model l2
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

from . import ccl

MIB = 1 << 20
SETTINGS = {
    # chiplets, L2 bytes per chiplet, tiles resident per chiplet
    "mi300x_like": dict(chiplets=4, l2_bytes=8 * MIB, slots=76),   # Sec. IV-A configuration
    "mi355x": dict(chiplets=8, l2_bytes=4 * MIB, slots=32),        # 8 XCDs x 32 CUs, 4 MB L2 each
}
PLACEMENTS = (
    ("rr_4k", ccl.CCL_PLACE_RR, 4096),
    ("rr_64k", ccl.CCL_PLACE_RR, 64 * 1024),
    ("rr_2m", ccl.CCL_PLACE_RR, 2 * MIB),
    ("coarse", ccl.CCL_PLACE_COARSE, 4096),
    ("ccl", ccl.CCL_PLACE_CCL, 4096),
)
WAYS = 16
LINE = 128
ELEM = {ccl.CCL_DT_FP8_E4M3: 1, ccl.CCL_DT_BF16: 2, ccl.CCL_DT_FP32: 4}


def k_step(ab_type: int) -> int:
    """K elements per model step: one 128-byte line of an A row."""
    return LINE // ELEM[ab_type]


def _remote(g, chiplets: int, grid_rows: int, placement: int, page: int, model: str,
            setting: dict, traversal: int, ab_type: int, c_type: int) -> int | None:
    try:
        plan = ccl.ccl_plan_typed(g.M, g.N, g.K, chiplets, grid_rows, page, ab_type, c_type)
    except ccl.CCLError as e:
        if e.status == 2:              # grid not tile-aligned for this GEMM
            return None
        raise
    mask = g.a_trans | (g.b_trans << 1)
    if model == "charge":
        return sum(ccl.ccl_remote_bytes(plan, placement, mask)["remote"])
    rec = ccl.ccl_remote_bytes_l2(plan, placement, mask, l2_bytes=setting["l2_bytes"],
                                  slots=setting["slots"], ways=WAYS, line_bytes=LINE,
                                  k_step=k_step(ab_type), traversal=traversal, threads=1)
    return sum(rec["remote"])


def evaluate(gemms, setting_name="mi300x_like", model: str = "l2", workers: int = 0,
             log=None, ab_type: int = ccl.CCL_DT_BF16, c_type: int = ccl.CCL_DT_BF16) -> list[dict]:
    """Best (grid, traversal) remote bytes of every GEMM under every placement.

    setting_name: a key of SETTINGS, or a dict with the same fields.
    ab_type / c_type: element types of A, B and of C (Fig. 7 data types).
    """
    setting = SETTINGS[setting_name] if isinstance(setting_name, str) else dict(setting_name)
    if not isinstance(setting_name, str):
        setting_name = "custom"
    G = setting["chiplets"]
    grids = [gr for gr in range(1, G + 1) if G % gr == 0]
    travs = (0, 1) if model == "l2" else (0,)
    jobs = [(gi, name, gr, tr) for gi in range(len(gemms)) for name, _, _ in PLACEMENTS
            for gr in grids for tr in travs]
    place = {name: (pl, page) for name, pl, page in PLACEMENTS}

    def run(job):
        gi, name, gr, tr = job
        pl, page = place[name]
        return job, _remote(gemms[gi], G, gr, pl, page, model, setting, tr, ab_type, c_type)

    best: dict = {}
    workers = workers or max(1, os.cpu_count() or 1)
    t0 = time.time()
    with ThreadPoolExecutor(max_workers=workers) as ex:          # ctypes calls release the GIL
        # largest GEMMs first so the pool stays busy
        order = sorted(jobs, key=lambda j: -gemms[j[0]].M * gemms[j[0]].N * gemms[j[0]].K)
        for (gi, name, gr, tr), rb in ex.map(run, order):
            if rb is None:
                continue
            key = (gi, name)
            if key not in best or (rb, gr, tr) < best[key]:
                best[key] = (rb, gr, tr)
    if log:
        log(f"{len(jobs)} configurations in {time.time() - t0:.1f} s")
    out = []
    for gi, g in enumerate(gemms):
        rec = {"gemm": g.name, "model": g.model, "tokens": g.tokens, "proj": g.proj, "pass": g.pass_,
               "M": g.M, "N": g.N, "K": g.K, "trans_a": g.a_trans, "trans_b": g.b_trans,
               "setting": setting_name, "traffic_model": model,
               "elem_bytes": [ELEM[ab_type], ELEM[ab_type], ELEM[c_type]]}
        if (gi, "ccl") not in best:        # no tile-aligned grid for this GEMM
            rec["no_aligned_grid"] = True
            out.append(rec)
            continue
        for name, _, _ in PLACEMENTS:
            rb, gr, tr = best[(gi, name)]
            rec[name] = {"remote_bytes": rb, "grid": f"{gr}x{G // gr}",
                         "traversal": ("rows", "cols")[tr]}
        rec["coarse_optimal"] = rec["coarse"]["remote_bytes"] <= rec["ccl"]["remote_bytes"]
        out.append(rec)
    return out


def _gmean(xs) -> float:
    return math.exp(sum(math.log(x) for x in xs) / len(xs)) if xs else float("nan")


def summarize(records: list[dict]) -> dict:
    """Per model: geometric means of placement / CCL and the fine-optimal count."""
    out = {}
    for model in sorted({r["model"] for r in records}):
        rs = [r for r in records if r["model"] == model and not r.get("no_aligned_grid")]
        s = {"gemms": len(rs), "fine_optimal": sum(not r["coarse_optimal"] for r in rs)}
        for name, _, _ in PLACEMENTS:
            if name == "ccl":
                continue
            ratios = [r[name]["remote_bytes"] / r["ccl"]["remote_bytes"] for r in rs
                      if r["ccl"]["remote_bytes"] > 0]
            s[f"{name}_over_ccl_gmean"] = _gmean(ratios)
            s[f"{name}_over_ccl_max"] = max(ratios) if ratios else float("nan")
        fine = [r for r in rs if not r["coarse_optimal"] and r["ccl"]["remote_bytes"] > 0]
        s["coarse_over_ccl_gmean_fine_optimal"] = _gmean(
            [r["coarse"]["remote_bytes"] / r["ccl"]["remote_bytes"] for r in fine])
        out[model] = s
    return out


def fig7(workers: int = 0, log=None) -> dict:
    """The sensitivity study of Fig. 7 in the finite-L2 model: mean remote
    bytes over the 12 GEMMs with 4K tokens (each placement at its best grid
    and traversal) while the per-chiplet L2 capacity varies with bf16
    operands, and while the data type varies with an 8 MB L2. Chiplets and
    resident tiles as in the MI300X-like setting."""
    import workloads as W

    gemms = [g for g in W.FFN_SWEEP if g.tokens == 4096]
    base = dict(SETTINGS["mi300x_like"])
    names = ("rr_4k", "coarse", "ccl")

    def mean_remote(setting, ab, c):
        recs = evaluate(gemms, setting, "l2", workers, log, ab, c)
        recs = [r for r in recs if not r.get("no_aligned_grid")]
        return {n: sum(r[n]["remote_bytes"] for r in recs) / len(recs) for n in names}

    out = {"gemms": len(gemms), "capacity_sweep_bf16": {}, "dtype_sweep_8mb": {}}
    for mb in (2, 4, 8, 16, 32):
        st = dict(base, l2_bytes=mb * MIB)
        out["capacity_sweep_bf16"][f"{mb}MB"] = mean_remote(st, ccl.CCL_DT_BF16, ccl.CCL_DT_BF16)
    for label, ab, c in (("fp8 (bf16 C)", ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_BF16),
                         ("bf16", ccl.CCL_DT_BF16, ccl.CCL_DT_BF16),
                         ("fp32", ccl.CCL_DT_FP32, ccl.CCL_DT_FP32)):
        out["dtype_sweep_8mb"][label] = mean_remote(dict(base, l2_bytes=8 * MIB), ab, c)
    return out


def markdown(records: list[dict]) -> str:
    cols = [name for name, _, _ in PLACEMENTS]
    lines = ["| GEMM | M×N×K | " + " | ".join(cols) + " | CCL grid | class |",
             "|" + "---|" * (len(cols) + 4)]
    for r in records:
        if r.get("no_aligned_grid"):
            lines.append(f"| {r['gemm']} | {r['M']}×{r['N']}×{r['K']} | no tile-aligned grid |")
            continue
        ccl_b = r["ccl"]["remote_bytes"]
        cells = []
        for c in cols:
            b = r[c]["remote_bytes"]
            cells.append(f"{b / 1e6:.1f} MB" + ("" if c == "ccl" or ccl_b == 0 else f" ({b / ccl_b:.2f}×)"))
        lines.append(f"| {r['gemm']} | {r['M']}×{r['N']}×{r['K']} | " + " | ".join(cells) +
                     f" | {r['ccl']['grid']} | {'coarse' if r['coarse_optimal'] else 'fine'} |")
    return "\n".join(lines)


def main(argv=None) -> int:
    import workloads as W

    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--setting", choices=sorted(SETTINGS), default="mi300x_like")
    ap.add_argument("--model", choices=("l2", "charge"), default="l2")
    ap.add_argument("--models", default="", help="comma-separated subset of FFN models")
    ap.add_argument("--tokens", default="", help="comma-separated subset of token counts")
    ap.add_argument("--workers", type=int, default=0)
    ap.add_argument("--out", default="", help="write the records and summary as JSON here")
    ap.add_argument("--markdown", action="store_true", help="print a markdown table")
    ap.add_argument("--fig7", action="store_true",
                    help="L2-capacity and data-type sensitivity (mean over the 4K-token GEMMs)")
    a = ap.parse_args(argv)
    if a.fig7:
        res = fig7(a.workers, log=lambda m: print(m, file=sys.stderr))
        if a.out:
            with open(a.out, "w") as f:
                json.dump(res, f, indent=1)
        print(json.dumps(res, indent=1))
        return 0
    gemms = list(W.FFN_SWEEP)
    if a.models:
        gemms = [g for g in gemms if g.model in a.models.split(",")]
    if a.tokens:
        gemms = [g for g in gemms if str(g.tokens) in a.tokens.split(",")]
    recs = evaluate(gemms, a.setting, a.model, a.workers, log=lambda m: print(m, file=sys.stderr))
    summ = summarize(recs)
    if a.out:
        with open(a.out, "w") as f:
            json.dump({"records": recs, "summary": summ}, f, indent=1)
    if a.markdown:
        print(markdown(recs))
    print(json.dumps(summ, indent=1))
    return 0


if __name__ == "__main__":
    sys.exit(main())
