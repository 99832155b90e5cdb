"""Throughput of the CCL GEMM hot path on one MI355X.

Workload (Llama-3.1-70B dense FFN forward, 8192 tokens, bf16, 8 chiplet
partitions on a 2x4 grid, 4 KB pages): one step is
    pack X (8192x8192, row-major -> CCL)
    H = X W_up        (8192x28672x8192, CCL GEMM)
    Y = H W_down      (8192x8192x28672, CCL GEMM; H is read in the CCL
                       layout the first GEMM wrote: same block grid)
    unpack Y (CCL -> row-major)
The weights are packed into CCL once before timing (load-time packing).
Inputs are synthetic (seeded, workloads module) and resident in HBM.

Prints one JSON line: value = GEMM TFLOP/s of the whole step, plus the
roofline of the dominant kernel (the GEMM, timed per launch with HIP events
on its stream), the remote-HBM-byte model for both GEMMs, and the CPU
oracle timed on a bounded sample (rank 0, one GPU only).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "CCL bf16 GEMM TFLOP/s (% MFMA peak); remote-HBM-byte reduction vs 4KB interleave"
PEAK_BF16_TFLOPS = 2516.6        # 256 CU x 4096 FLOP/clk x 2.4 GHz (dense)
PEAK_FP8_TFLOPS = 5033.2         # 256 CU x 8192 FLOP/clk x 2.4 GHz (dense fp8)
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_llama_fwd_traffic.json")
CSRC = os.path.join(ROOT, "paper_2606_11718_amd", "csrc")
# the sources that fix the GEMM's memory traffic: the kernels, the
# workgroup -> tile map and the plan that picks tile shape and raster
GEMM_SRCS = tuple(os.path.join(CSRC, f) for f in ("kernels/gemm.hip", "host/tile_map.hpp", "host/plan.cpp"))


def kernel_hash(srcs=GEMM_SRCS) -> str:
    """Hash of the GEMM sources with comments and whitespace removed, so that
    only a change to the code itself retires the committed counters."""
    import re
    h = hashlib.sha256()
    for src in srcs:
        text = open(src, encoding="utf-8").read()
        text = re.sub(r"//[^\n]*", "", text)
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


# (M K + K N + M N) * 2 bytes of either Llama forward GEMM
ALGO_BYTES = (8192 * 8192 + 2 * 8192 * 28672) * 2


def measured_traffic(launch_flops_unused=None):
    """Bytes per GEMM launch between L2 and memory (reads and writes) from
    the committed rocprofv3 counter runs, if they were taken on the current
    kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    t = json.load(open(TRAFFIC_FILE))
    if t.get("kernel_hash") != kernel_hash():
        return None
    return t.get("hbm_bytes_per_launch")


_SMI = {}


def smi_sample():
    """One reading of socket power (W) and the XCD clocks (MHz), in-process
    through the amdsmi library (no subprocess)."""
    try:
        import amdsmi
        if "h" not in _SMI:
            amdsmi.amdsmi_init(amdsmi.AmdSmiInitFlags.INIT_AMD_GPUS)
            _SMI["h"] = amdsmi.amdsmi_get_processor_handles()[0]
        m = amdsmi.amdsmi_get_gpu_metrics_info(_SMI["h"])
        power = m.get("current_socket_power")
        clocks = [c for c in (m.get("current_gfxclks") or []) if isinstance(c, int) and c > 0]
        if not isinstance(power, (int, float)) or not clocks:
            return None
        return float(power), clocks
    except Exception:
        return None


def sustained_clock(step, seconds: float):
    """Run `step` back to back for `seconds` and sample power and clocks
    from a second thread (after a 1 s ramp)."""
    import statistics
    import threading
    import torch
    stop = time.time() + seconds
    samples = []

    def sampler():
        time.sleep(1.0)
        while time.time() < stop - 0.5:
            v = smi_sample()
            if v:
                samples.append(v)
            time.sleep(0.3)

    th = threading.Thread(target=sampler)
    th.start()
    while time.time() < stop:
        for _ in range(10):
            step(False)
        torch.cuda.synchronize()
    th.join()
    if not samples:
        return None
    clk = statistics.median([c for _, cs in samples for c in cs])
    return {"gfx_clock_mhz_median": clk, "socket_power_w_median": statistics.median([p for p, _ in samples]),
            "samples": len(samples)}


def cpu_baseline(target_s: float):
    """The oracle's fp64 GEMMs of the step (up and down projections) on a
    row sample sized for about target_s seconds (the whole GEMMs if the host
    is fast enough). The bf16 operands are widened to float64 once, outside
    the timed calls; the timed calls are the oracle's GEMM."""
    import threadpoolctl
    import workloads as W
    from oracle import gemm as OG

    wl, g_up = W.gemm_by_name("llama_up")
    _, g_dn = W.gemm_by_name("llama_down")
    ops = []
    for g in (g_up, g_dn):
        ops.append((W.draw(wl.tensors[g.a_src]), OG.decode_bf16(W.draw(wl.tensors[g.b_src]))))
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])

    def run(rows):
        t = 0.0
        for A_bits, B in ops:
            A = OG.decode_bf16(A_bits[:rows])
            t0 = time.perf_counter()
            OG.gemm_fp64(A, B)
            t += time.perf_counter() - t0
        return t

    run(32)                                   # warm the BLAS threads
    t_cal = run(128)
    rows = int(min(g_up.M, 128 * target_s / max(t_cal, 1e-3)))
    rows = max(128, (rows // 64) * 64)
    t = run(rows)
    flops = 2.0 * rows * (g_up.N * g_up.K + g_dn.N * g_dn.K)
    blas = [f"{i.get('internal_api')} {i.get('version')} ({i.get('num_threads')} threads)"
            for i in info if i.get("user_api") == "blas"]
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"fp64 oracle GEMMs (numpy BLAS) of the step, first {rows} of 8192 token rows "
                      f"of X W_up and H W_down: {flops / 1e12:.3f} TFLOP in {t:.2f} s",
            "cpu_model": _cpu_model(), "host_cpus": len(os.sched_getaffinity(0)), "blas": blas,
            "other_oracle_parts": _oracle_other_parts(ops[0][0])}


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo", encoding="utf-8"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_other_parts(X_bits):
    """The oracle's CCL pack of X (numpy reshape/transpose, 8192 x 8192 bf16,
    2 x 4 grid) and its remote-byte model under each placement on the Qwen3
    gate/up shape (4096 x 1536 x 2048, 2 x 4 grid, 4 KB pages), each timed
    once on the host."""
    from oracle import layout as OL
    from oracle import traffic as OT
    t0 = time.perf_counter()
    OL.pack_reshape(X_bits, 2, 4, 4096)
    t_pack = time.perf_counter() - t0
    model = {}
    for name, pl in (("rr", OT.RR), ("coarse", OT.COARSE), ("ccl", OT.CCL)):
        t0 = time.perf_counter()
        OT.remote_bytes(4096, 1536, 2048, 2, 4, 4096, pl)
        model[name] = round(time.perf_counter() - t0, 3)
    return {"pack_X_GBs": round(2 * X_bits.nbytes / t_pack / 1e9, 2),
            "byte_model_qwen_gate_up_s": model}


def compare_layouts(reps: int, sustained: float = 0.0, rounds: int = 1):
    """Per-launch time of the same GEMM kernel under three operand layouts /
    tile maps on the Llama FFN forward shapes: CCL operands with the
    XCD-aware map (ccl_gemm), row-major operands with native dispatch, and
    row-major operands with the XCD-aware map (ccl_gemm_rowmajor). The
    XCD-aware map runs at both raster group heights (4 and 8 tile rows), so
    each layout can be compared at its best; `plan_group_m` is the height
    the plan picks by itself. With `sustained` > 0 each variant first runs
    back to back for that many seconds, so the power-limited clock settles
    at its own level; `rounds` > 1 alternates the variants that many times
    and reports every round's median."""
    import numpy as np
    import torch
    from paper_2606_11718_amd import ccl

    out = {}
    for name, (M, N, K) in (("llama_up", (8192, 28672, 8192)), ("llama_down", (8192, 8192, 28672))):
        plans = {}
        for gm in (4, 8):
            old = os.environ.get("CCL_GEMM_GROUP_M")
            os.environ["CCL_GEMM_GROUP_M"] = str(gm)
            try:
                plans[gm] = ccl.ccl_plan(M, N, K, 8, 2, 4096)
            finally:
                if old is None:
                    os.environ.pop("CCL_GEMM_GROUP_M", None)
                else:
                    os.environ["CCL_GEMM_GROUP_M"] = old
        g = torch.Generator(device="cuda").manual_seed(7)
        A = (torch.randn(M * K, device="cuda", generator=g)).to(torch.bfloat16)
        B = (torch.randn(K * N, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
        C = torch.empty(M * N, device="cuda", dtype=torch.bfloat16)
        st = torch.cuda.current_stream()
        # One pack of A (a copy of 2*M*K*2 known bytes) before the GEMMs: a
        # reference for the memory counters of the same run.
        Ac = torch.empty(M * K, device="cuda", dtype=torch.bfloat16)
        ccl.ccl_pack(plans[4], ccl.CCL_A, A, K, 0, Ac, st)
        torch.cuda.synchronize()
        del Ac
        variants = {
            "ccl_remap_g4": lambda: ccl.ccl_gemm(plans[4], A, B, C, st),
            "ccl_remap_g8": lambda: ccl.ccl_gemm(plans[8], A, B, C, st),
            "rowmajor_native": lambda: ccl.ccl_gemm_rowmajor(plans[4], A, B, C, 0, st),
            "rowmajor_remap_g4": lambda: ccl.ccl_gemm_rowmajor(plans[4], A, B, C, 1, st),
            "rowmajor_remap_g8": lambda: ccl.ccl_gemm_rowmajor(plans[8], A, B, C, 1, st),
        }
        res = {}
        for rnd in range(rounds):
            for vname, fn in variants.items():
                for _ in range(3):
                    fn()
                torch.cuda.synchronize()
                t_end = time.time() + sustained
                while time.time() < t_end:
                    for _ in range(5):
                        fn()
                    torch.cuda.synchronize()
                ts = []
                for _ in range(reps):
                    e0, e1 = torch.cuda.Event(True), torch.cuda.Event(True)
                    e0.record(st)
                    fn()
                    e1.record(st)
                    ts.append((e0, e1))
                torch.cuda.synchronize()
                ms = float(np.median([a.elapsed_time(b) for a, b in ts]))
                tf = round(2 * M * N * K / ms / 1e9, 1)
                if rounds == 1:
                    res[vname] = {"ms": round(ms, 4), "tflops": tf}
                else:
                    res.setdefault(vname, {"tflops_by_round": []})["tflops_by_round"].append(tf)
        default = ccl.ccl_plan(M, N, K, 8, 2, 4096)
        res["plan_group_m"] = next(gm for gm in (4, 8) if all(
            ccl.ccl_debug_tile_of_wg(default, w) == ccl.ccl_debug_tile_of_wg(plans[gm], w) for w in range(0, 4096, 7)))
        out[name] = res
    return out


def operand_diagnostic(reps: int, seconds: float):
    """A diagnostic, not the metric: the Llama forward GEMMs (CCL operands,
    the plan's tile map) on all-zero operands and on random operands of the
    benchmark's distributions, in the same buffers. Zero operands hardly
    toggle the datapaths, so the GPU keeps its top clock below the socket
    power limit; with random operands the limit sets the clock. Per variant:
    the median per-launch time over `reps` launches, then `seconds` of
    back-to-back launches with the sampled clock and power."""
    import numpy as np
    import torch
    from paper_2606_11718_amd import ccl

    out = {}
    for name, (M, N, K) in (("llama_up", (8192, 28672, 8192)), ("llama_down", (8192, 8192, 28672))):
        plan = ccl.ccl_plan(M, N, K, 8, 2, 4096)
        g = torch.Generator(device="cuda").manual_seed(11)
        Ar = torch.randn(M * K, device="cuda", generator=g).to(torch.bfloat16)
        Br = (torch.randn(K * N, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
        Az, Bz = torch.zeros_like(Ar), torch.zeros_like(Br)
        C = torch.empty(M * N, device="cuda", dtype=torch.bfloat16)
        st = torch.cuda.current_stream()
        res = {}
        for data, (A, B) in (("zero", (Az, Bz)), ("random", (Ar, Br))):
            def step(_timed, A=A, B=B):
                ccl.ccl_gemm(plan, A, B, C, st)
            for _ in range(5):
                step(False)
            torch.cuda.synchronize()
            ev = [(torch.cuda.Event(True), torch.cuda.Event(True)) for _ in range(reps)]
            for e0, e1 in ev:
                e0.record(st)
                step(True)
                e1.record(st)
            torch.cuda.synchronize()
            ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))
            rec = {"ms": round(ms, 4), "tflops": round(2 * M * N * K / ms / 1e9, 1),
                   "frac": round(2 * M * N * K / ms / 1e9 / PEAK_BF16_TFLOPS, 4)}
            if seconds > 0:
                clk = sustained_clock(step, seconds)
                if clk:
                    rec["sustained"] = clk
            res[data] = rec
        out[name] = res
        del Ar, Br, Az, Bz, C
    return out


def remote_report():
    """Remote-byte model (the library's host model) for every workload GEMM,
    grid and page size: totals per placement, floor, excess over the floor,
    RR/CCL and COARSE/CCL ratios; geomean of best-of-grid ratios per model
    family (best-of-grid: min over grids per placement, as the paper keeps
    the best partition per placement)."""
    import math
    import workloads as W
    from paper_2606_11718_amd import ccl

    rows, best = [], {}
    for wl in W.WORKLOADS.values():
        for g in wl.gemms:
            grids = g.grids if g.grids != (0,) else (0,)
            for gr in grids:
                for P in g.pages:
                    plan = ccl.ccl_plan(g.M, g.N, g.K, g.chiplets, gr, P)
                    Gr, Gc = ccl.ccl_plan_grid(plan)
                    rec = {}
                    for name, code in (("rr", ccl.CCL_PLACE_RR), ("coarse", ccl.CCL_PLACE_COARSE),
                                       ("ccl", ccl.CCL_PLACE_CCL)):
                        r = ccl.ccl_remote_bytes(plan, code, g.a_trans | (g.b_trans << 1))
                        rec[name] = sum(r["remote"])
                        rec["floor"] = r["floor"]
                        rec["accessed"] = sum(r["accessed"])
                    row = {"gemm": g.name, "MNK": f"{g.M}x{g.N}x{g.K}", "grid": f"{Gr}x{Gc}", "page": P,
                           **rec, "excess_rr": rec["rr"] - rec["floor"], "excess_coarse": rec["coarse"] - rec["floor"],
                           "excess_ccl": rec["ccl"] - rec["floor"],
                           "rr_over_ccl": rec["rr"] / rec["ccl"] if rec["ccl"] else None,
                           "coarse_over_ccl": rec["coarse"] / rec["ccl"] if rec["ccl"] else None}
                    rows.append(row)
                    key = (g.name, P)
                    b = best.setdefault(key, {"rr": None, "coarse": None, "ccl": None})
                    for pl in ("rr", "coarse", "ccl"):
                        b[pl] = rec[pl] if b[pl] is None else min(b[pl], rec[pl])
    fam = {"qwen": [], "llama": []}
    for (name, P), b in best.items():
        if P != 4096 or name == "tiny":
            continue
        fam["qwen" if name.startswith("qwen") else "llama"].append((b["rr"] / b["ccl"], b["coarse"] / b["ccl"]))
    geo = {f: {"rr_over_ccl": math.exp(sum(math.log(x) for x, _ in v) / len(v)),
               "coarse_over_ccl": math.exp(sum(math.log(y) for _, y in v) / len(v)), "gemms": len(v)}
           for f, v in fam.items() if v}
    return {"rows": rows, "best_of_grid_geomean_4k": geo}


def fp8_gemms(reps: int):
    """Per-launch time of the fp8 (E4M3) CCL GEMM on the Llama FFN forward
    shapes (bf16 C), the same kernel structure at twice the MFMA rate per K."""
    import numpy as np
    import torch
    from paper_2606_11718_amd import ccl

    out = {}
    for name, (M, N, K) in (("llama_up", (8192, 28672, 8192)), ("llama_down", (8192, 8192, 28672))):
        plan = ccl.ccl_plan_typed(M, N, K, 8, 2, 4096, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_BF16)
        g = torch.Generator(device="cuda").manual_seed(11)
        A = torch.randn(M * K, device="cuda", generator=g).to(torch.float8_e4m3fn).view(torch.uint8)
        B = torch.randn(K * N, device="cuda", generator=g).to(torch.float8_e4m3fn).view(torch.uint8)
        C = torch.empty(M * N, device="cuda", dtype=torch.bfloat16)
        st = torch.cuda.current_stream()
        # half a second of back-to-back launches first, so the clock has
        # settled at this kernel's power level before timing
        t_end = time.time() + 0.5
        while time.time() < t_end:
            for _ in range(10):
                ccl.ccl_gemm(plan, A, B, C, st)
            torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(True), torch.cuda.Event(True)
            e0.record(st)
            ccl.ccl_gemm(plan, A, B, C, st)
            e1.record(st)
            ts.append((e0, e1))
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in ts]))
        tf = 2 * M * N * K / ms / 1e9
        out[name] = {"ms": round(ms, 4), "tflops": round(tf, 1),
                     "frac_of_fp8_peak": round(tf / PEAK_FP8_TFLOPS, 4)}
        del A, B, C
    out["peak"] = PEAK_FP8_TFLOPS
    out["kernel"] = ("gemm_fp8p_kernel (256x256, 8 waves, v_mfma_f32_16x16x128_f8f6f4, 128-wide K "
                     "steps, 3 A and 2 B LDS stages, fragment reads pipelined across steps)")
    return out


def pack_hbm(reps: int):
    """HBM rate of the pack kernels on the Llama-3.1-70B operands, each
    timed alone: the row-major packs of the forward pass (X, W_up), the
    stored-transpose packs of the backward pass (X^T as A of dW_up = X^T dY,
    W_up^T as B of dX = dY W_up^T, both on the 1x8 grid) and the unpack of
    Y. Tensors smaller than the 256 MB Infinity Cache rotate over buffer
    sets of more than 1 GB in total, so every launch reads and writes HBM.
    Bytes = read + write of the logical tensor (padding is never written)."""
    import torch
    from paper_2606_11718_amd import ccl

    cases = [
        # name, plan (M, N, K, Gr), operand, stored rows x cols, transposed, unpack
        ("pack_X", (8192, 28672, 8192, 2), ccl.CCL_A, (8192, 8192), 0, False),
        ("pack_W_up", (8192, 28672, 8192, 2), ccl.CCL_B, (8192, 28672), 0, False),
        ("pack_trans_X_T", (8192, 28672, 8192, 1), ccl.CCL_A, (8192, 8192), 1, False),
        ("pack_trans_W_up_T", (8192, 8192, 28672, 1), ccl.CCL_B, (8192, 28672), 1, False),
        ("unpack_Y", (8192, 8192, 28672, 2), ccl.CCL_C, (8192, 8192), 0, True),
    ]
    st = torch.cuda.current_stream()
    out = {}
    for name, (M, N, K, gr), op, (sr, sc), trans, unpack in cases:
        plan = ccl.ccl_plan(M, N, K, 8, gr, 4096)
        lay = ccl.ccl_plan_layout(plan, op)
        nbytes = sr * sc * 2
        sets = 1 if nbytes > (256 << 20) else (1 << 30) // nbytes + 1
        rm = [torch.empty(sr * sc, dtype=torch.int16, device="cuda") for _ in range(sets)]
        cc = [torch.empty(lay.total_bytes // 2, dtype=torch.int16, device="cuda") for _ in range(sets)]
        if unpack:
            calls = [(lambda r=r, c=c: ccl.ccl_unpack(plan, op, c, r, sc, st)) for r, c in zip(rm, cc)]
        else:
            calls = [(lambda r=r, c=c: ccl.ccl_pack(plan, op, r, sc, trans, c, st)) for r, c in zip(rm, cc)]
        for c in calls[:3]:
            c()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(True), torch.cuda.Event(True)
        n = max(reps, 2 * sets)
        e0.record(st)
        for i in range(n):
            calls[i % sets]()
        e1.record(st)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        gbs = 2 * nbytes / (ms * 1e-3) / 1e9
        out[name] = {"MB": round(nbytes / 1e6, 1), "buffer_sets": sets, "ms": round(ms, 4),
                     "GBs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
        del rm, cc, calls
        torch.cuda.empty_cache()
    out["peak"] = PEAK_HBM_GBS
    return out


# One GPU's share of the Llama-3.1-70B FFN under 8-way tensor parallelism:
# the up projection split by output columns (W_up 8192 x 28672/8), the down
# projection by its K (W_down 28672/8 x 8192), each GEMM at full token
# count. The path would shard this way over 8 GPUs; one GPU runs its share.
TP8_SHARDS = (("llama_up_tp8_shard", 8192, 28672 // 8, 8192),
              ("llama_down_tp8_shard", 8192, 8192, 28672 // 8))


def _time_ccl_and_vendor(name, M, N, K, G, grid_rows, reps):
    """ccl_gemm on random operands already in CCL (plan at grid_rows, 4 KB
    pages) and torch.matmul of row-major operands of the same shape, each
    timed as reps back-to-back launches after 3 warm-up ones; plus the
    library's split-K choice where it takes more than one range."""
    import torch
    from paper_2606_11718_amd import ccl

    flops = 2 * M * N * K
    plan = ccl.ccl_plan(M, N, K, G, grid_rows, 4096)
    gr, gc = ccl.ccl_plan_grid(plan)
    lay = [ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C)]
    gen = torch.Generator(device="cuda").manual_seed(5)
    A = torch.randn(lay[0].total_bytes // 2, device="cuda", generator=gen).to(torch.bfloat16)
    B = (torch.randn(lay[1].total_bytes // 2, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    C = torch.empty(lay[2].total_bytes // 2, device="cuda", dtype=torch.bfloat16)
    st = torch.cuda.current_stream()

    def timed(call):
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(True), torch.cuda.Event(True)
        e0.record(st)
        for _ in range(reps):
            call()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    ms = timed(lambda: ccl.ccl_gemm(plan, A, B, C, st))
    tm, tn, _ = ccl.ccl_debug_gemm_config(plan)
    rec = {"MNK": f"{M}x{N}x{K}", "grid": f"{gr}x{gc}", "tile": f"{tm}x{tn}",
           "ms": round(ms, 4), "tflops": round(flops / ms / 1e9, 1)}
    # the vendor library on the same shape, box and power limit:
    # torch.matmul of contiguous row-major bf16 operands
    Ar = torch.randn(M, K, device="cuda", generator=gen).to(torch.bfloat16)
    Br = (torch.randn(K, N, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    Cr = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
    ms_v = timed(lambda: torch.matmul(Ar, Br, out=Cr))
    rec["vendor_matmul"] = {"ms": round(ms_v, 4), "tflops": round(flops / ms_v / 1e9, 1),
                            "ccl_speedup": round(ms_v / ms, 3),
                            "blas": str(torch.backends.cuda.preferred_blas_library())}
    del Ar, Br, Cr
    ranges, ws_bytes = ccl.ccl_gemm_splitk_workspace(plan, 0)
    if ranges > 1:             # the library's split-K choice for this shape
        ws = torch.empty(ws_bytes, device="cuda", dtype=torch.uint8)
        ms_s = timed(lambda: ccl.ccl_gemm_splitk(plan, 1.0, A, B, 0.0, C, ranges, ws,
                                                 ws_bytes, st))
        rec["splitk"] = {"ranges": ranges, "ms": round(ms_s, 4),
                         "tflops": round(flops / ms_s / 1e9, 1)}
        del ws
    del A, B, C
    return rec


def workload_gemms(reps: int):
    """Per-launch time of ccl_gemm on every workload GEMM shape (bf16, random
    operands already in CCL), at the grid the parity tests use: the small
    Qwen3 shapes, the tiny case and the Llama backward GEMMs; then one GPU's
    share of the Llama FFN under 8-way tensor parallelism (TP8_SHARDS, the
    plan's automatic grid). Beside each, torch.matmul of row-major operands
    of the same shape (the vendor BLAS, free to use every CU) timed the same
    way."""
    import workloads as W

    out = {}
    for wl in W.WORKLOADS.values():
        for g in wl.gemms:
            out[g.name] = _time_ccl_and_vendor(g.name, g.M, g.N, g.K, g.chiplets, g.grids[0], reps)
    for name, M, N, K in TP8_SHARDS:
        out[name] = _time_ccl_and_vendor(name, M, N, K, 8, 0, reps)
    return out


def gemm_timeline(reps: int):
    """Phase timeline of the bf16 GEMM on every workload shape and the Llama
    forward pair (ccl_debug_gemm_timeline: per-wave real-time counter at
    start, after the prologue, after the K loop, after the stores' issue;
    shader clock over the loop). reps launches back to back after 3 warm-up
    launches; medians over those launches of per-launch figures."""
    import numpy as np
    import torch
    import workloads as W
    from paper_2606_11718_amd import ccl

    out = {}
    names = ["tiny", "qwen_gate_up", "qwen_dW_down", "qwen_dH", "llama_up", "llama_down"]
    for name in names:
        _, g = W.gemm_by_name(name)
        plan = ccl.ccl_plan(g.M, g.N, g.K, g.chiplets, g.grids[0], 4096)
        tm, tn, wgs = ccl.ccl_debug_gemm_config(plan)
        lay = [ccl.ccl_plan_layout(plan, op) for op in (ccl.CCL_A, ccl.CCL_B, ccl.CCL_C)]
        gen = torch.Generator(device="cuda").manual_seed(5)
        A = torch.randn(lay[0].total_bytes // 2, device="cuda", generator=gen).to(torch.bfloat16)
        B = (torch.randn(lay[1].total_bytes // 2, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
        C = torch.empty(lay[2].total_bytes // 2, device="cuda", dtype=torch.bfloat16)
        words = wgs * 8 * 8
        tl = torch.zeros(reps * words, dtype=torch.int64, device="cuda")
        st = torch.cuda.current_stream()
        for _ in range(3):
            ccl.ccl_gemm(plan, A, B, C, st)
        for r in range(reps):
            ccl.ccl_debug_gemm_timeline(plan, A, B, C, tl[r * words:], words * 8, st)
        torch.cuda.synchronize()
        rec = tl.cpu().numpy().reshape(reps, wgs, 8, 8)
        live = rec[:, :, 0, 0] > 0
        steps = g.K // 32
        flop_per_step = 2 * tm * tn * 32
        per = []
        for r in range(reps):
            x = rec[r][live[r]]                       # (live wgs, 8 waves, 8 words)
            t0 = x[:, :, 0].min(1)
            t1, t2, t3 = x[:, :, 1].max(1), x[:, :, 2].max(1), x[:, :, 3].max(1)
            ghz = (x[:, 0, 5] - x[:, 0, 4]) / ((x[:, 0, 2] - x[:, 0, 0]) * 10.0)
            loop_us = (t2 - t1) / 100.0
            # gap between consecutive tiles on one CU: the next workgroup's
            # start after the previous one's last store was issued
            cu = x[:, 0, 6] * 65536 + (x[:, 0, 7] & 0xFF00)
            gaps = []
            for c in np.unique(cu):
                sel = np.where(cu == c)[0]
                if len(sel) > 1:
                    o = sel[np.argsort(t0[sel])]
                    gaps.extend((t0[o[1:]] - t3[o[:-1]]).tolist())
            per.append({
                "tile_gap_us": float(np.median(gaps)) / 100.0 if gaps else 0.0,
                "span_us": (t3.max() - t0.min()) / 100.0,
                # until the first min(workgroups, 256) workgroups (one per CU) started
                "dispatch_us": (np.sort(t0)[min(len(t0), 256) - 1] - t0.min()) / 100.0,
                "prologue_us": float(np.median(t1 - t0)) / 100.0,
                "loop_us": float(np.median(loop_us)),
                "epilogue_us": float(np.median(t3 - t2)) / 100.0,
                "loop_clock_ghz": float(np.median(ghz)),
                "loop_mfma_frac": float(np.median(flop_per_step / 4096.0 * steps
                                                  / (loop_us * 1e3 * ghz))),
            })
        med = {k: round(float(np.median([p_[k] for p_ in per])), 3) for k in per[0]}
        med.update({"MNK": f"{g.M}x{g.N}x{g.K}", "tile": f"{tm}x{tn}", "workgroups": wgs,
                    "k_steps": steps, "launches": reps})
        out[name] = med
        del A, B, C, tl
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--remote-report", action="store_true",
                    help="only print the remote-byte model report (host only, no GPU)")
    ap.add_argument("--compare-layouts", action="store_true",
                    help="only time CCL vs row-major operands and tile maps, print one JSON line")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--sustained", type=float, default=0.0,
                    help="--compare-layouts: seconds of back-to-back launches before timing each variant")
    ap.add_argument("--rounds", type=int, default=1,
                    help="--compare-layouts: alternate the variants this many times")
    ap.add_argument("--operand-diagnostic", action="store_true",
                    help="only time the Llama GEMMs on zero vs random operands (a diagnostic of the "
                         "power limit, not the metric), print one JSON line")
    ap.add_argument("--no-fp8", action="store_true", help="skip the fp8 GEMM timing")
    ap.add_argument("--fp8-only", action="store_true",
                    help="only time the fp8 GEMMs, print one JSON line")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip timing the GEMM of every workload shape")
    ap.add_argument("--workloads-only", action="store_true",
                    help="only time the GEMM of every workload shape, print one JSON line")
    ap.add_argument("--gemm-timeline", action="store_true",
                    help="only record the per-workgroup phase timeline of the bf16 GEMM on the "
                         "workload shapes, print one JSON line")
    ap.add_argument("--no-pack-hbm", action="store_true",
                    help="skip timing the pack kernels alone on rotating buffers")
    ap.add_argument("--clock-seconds", type=float, default=4.0,
                    help="sustained run after the timed steps that samples clock/power (0: off)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested); the CCL GEMM "
              "path here has no multi-GPU sharding.", file=sys.stderr)
        sys.exit(2)

    if args.remote_report:
        print(json.dumps(remote_report()), flush=True)
        return

    import numpy as np
    import torch

    import workloads as W
    from paper_2606_11718_amd import ccl

    if args.compare_layouts:
        print(json.dumps({"compare_layouts": compare_layouts(args.reps, args.sustained, args.rounds)}),
              flush=True)
        return
    if args.operand_diagnostic:
        print(json.dumps({"operand_diagnostic": operand_diagnostic(args.reps, args.clock_seconds)}),
              flush=True)
        return
    if args.fp8_only:
        print(json.dumps({"fp8_gemm": fp8_gemms(args.reps)}), flush=True)
        return
    if args.workloads_only:
        print(json.dumps({"workload_gemms": workload_gemms(args.reps)}), flush=True)
        return
    if args.gemm_timeline:
        print(json.dumps({"gemm_timeline": gemm_timeline(args.reps)}), flush=True)
        return

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = W.WORKLOADS["llama_fwd"]
    _, g_up = W.gemm_by_name("llama_up")
    _, g_dn = W.gemm_by_name("llama_down")
    P, G, Gr = 4096, 8, 2
    plan_up = ccl.ccl_plan(g_up.M, g_up.N, g_up.K, G, Gr, P)
    plan_dn = ccl.ccl_plan(g_dn.M, g_dn.N, g_dn.K, G, Gr, P)
    L = {name: ccl.ccl_plan_layout(p, op) for name, p, op in
         (("X", plan_up, ccl.CCL_A), ("Wup", plan_up, ccl.CCL_B), ("H", plan_up, ccl.CCL_C),
          ("Hin", plan_dn, ccl.CCL_A), ("Wdn", plan_dn, ccl.CCL_B), ("Y", plan_dn, ccl.CCL_C))}
    # the up GEMM's C layout is the down GEMM's A layout (same grid over 8192 x 28672)
    assert L["H"] == L["Hin"]

    def dev_bits(t):
        return torch.from_numpy(W.draw(wl.tensors[t]).view(np.int16)).to(dev)

    def empty(lay):
        return torch.empty(lay.total_bytes // 2, dtype=torch.int16, device=dev)

    X = dev_bits("X")
    Wup_c, Wdn_c = empty(L["Wup"]), empty(L["Wdn"])
    w = dev_bits("W_up")
    ccl.ccl_pack(plan_up, ccl.CCL_B, w, g_up.N, 0, Wup_c)
    torch.cuda.synchronize()
    del w
    w = dev_bits("W_down")
    ccl.ccl_pack(plan_dn, ccl.CCL_B, w, g_dn.N, 0, Wdn_c)
    torch.cuda.synchronize()
    del w
    Xc, Hc, Yc = empty(L["X"]), empty(L["H"]), empty(L["Y"])
    Y = torch.empty(g_dn.M, g_dn.N, dtype=torch.int16, device=dev)

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    marks = []

    def step(timed):
        e = [ev() for _ in range(5)] if timed else None
        if timed:
            e[0].record(stream)
        ccl.ccl_pack(plan_up, ccl.CCL_A, X, g_up.K, 0, Xc, stream)
        if timed:
            e[1].record(stream)
        ccl.ccl_gemm(plan_up, Xc, Wup_c, Hc, stream)
        if timed:
            e[2].record(stream)
        ccl.ccl_gemm(plan_dn, Hc, Wdn_c, Yc, stream)
        if timed:
            e[3].record(stream)
        ccl.ccl_unpack(plan_dn, ccl.CCL_C, Yc, Y, g_dn.N, stream)
        if timed:
            e[4].record(stream)
            marks.append(e)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0, t1 = ev(), ev()
    t0.record(stream)
    for _ in range(args.steps):
        step(True)
    t1.record(stream)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_step = total_ms / args.steps
    per = {"pack_x": [], "gemm_up": [], "gemm_down": [], "unpack_y": []}
    for e in marks:
        per["pack_x"].append(e[0].elapsed_time(e[1]))
        per["gemm_up"].append(e[1].elapsed_time(e[2]))
        per["gemm_down"].append(e[2].elapsed_time(e[3]))
        per["unpack_y"].append(e[3].elapsed_time(e[4]))
    avg = {k: float(np.mean(v)) for k, v in per.items()}

    gemm_flops = float(g_up.flops)                  # = g_dn.flops
    step_flops = g_up.flops + g_dn.flops
    value = step_flops / (ms_step * 1e-3) / 1e12
    gemm_ms = (avg["gemm_up"] + avg["gemm_down"]) / 2
    achieved = gemm_flops / (gemm_ms * 1e-3) / 1e12
    traffic = measured_traffic()
    copy_bytes = 2 * 8192 * 8192 * 2                # read + write of X (or Y)

    remote = {}
    for name, p, g in (("llama_up", plan_up, g_up), ("llama_down", plan_dn, g_dn)):
        r = {pl: sum(ccl.ccl_remote_bytes(p, code, 0)["remote"])
             for pl, code in (("rr_4k", ccl.CCL_PLACE_RR), ("coarse_4k", ccl.CCL_PLACE_COARSE),
                              ("ccl_4k", ccl.CCL_PLACE_CCL))}
        r["rr_over_ccl"] = round(r["rr_4k"] / r["ccl_4k"], 4)
        r["coarse_over_ccl"] = round(r["coarse_4k"] / r["ccl_4k"], 4)
        remote[name] = r

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama_fwd: Llama-3.1-70B-like FFN forward, X[8192x8192] W_up[8192x28672] "
                               "then H W_down[28672x8192], 8 XCD partitions on a 2x4 grid, 4 KB pages",
                   "tokens": 8192, "grid": "2x4", "chiplets": G, "page_bytes": P,
                   "gemm_tile": list(ccl.ccl_debug_gemm_config(plan_up)[:2])},
        "pct_mfma_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic,
                     "traffic_counts": ("bytes per launch between the XCDs' L2 and memory (DRAM-class "
                                        "read requests x 128 B + write bytes), from committed rocprofv3 "
                                        "passes on this kernel source; the Infinity Cache is on that "
                                        "path, so an upper bound on HBM bytes"),
                     "algorithmic_bytes": ALGO_BYTES,
                     "traffic_over_algorithmic": (round(traffic / ALGO_BYTES, 3) if traffic else None),
                     "kernel": ("gemm_kernel<256,256,8 waves> (up and down launches)"
                                if os.environ.get("CCL_GEMM_A_PAIRS") == "0" else
                                "gemm_a2_kernel (256x256, 8 waves, A staged in 64-K pairs; up and "
                                "down launches)"),
                     "avg_launch_ms": round(gemm_ms, 4),
                     "launch_ms": {g: {"mean": round(avg[g], 4), "median": round(float(np.median(per[g])), 4),
                                       "min": round(float(np.min(per[g])), 4)} for g in ("gemm_up", "gemm_down")}},
        "kernels_ms": {k: round(v, 4) for k, v in avg.items()},
        "copy_roofline": {"bound": "hbm", "unit": "GB/s", "peak": PEAK_HBM_GBS,
                          "pack_x": round(copy_bytes / (avg["pack_x"] * 1e-3) / 1e9, 1),
                          "unpack_y": round(copy_bytes / (avg["unpack_y"] * 1e-3) / 1e9, 1)},
        "remote_bytes": remote,
    }
    if args.clock_seconds > 0:
        clk = sustained_clock(step, args.clock_seconds)
        if clk:
            clk["clock_adjusted_peak_tflops"] = round(PEAK_BF16_TFLOPS * clk["gfx_clock_mhz_median"] / 2400.0, 1)
            clk["gemm_frac_of_clock_adjusted_peak"] = round(achieved / clk["clock_adjusted_peak_tflops"], 4)
        out["sustained_clock"] = clk
    del X, Wup_c, Wdn_c, Xc, Hc, Yc, Y
    torch.cuda.empty_cache()
    if not args.no_fp8:
        out["fp8_gemm"] = fp8_gemms(args.reps)
    if not args.no_pack_hbm:
        out["pack_hbm"] = pack_hbm(args.reps)
    if not args.no_workloads:
        out["workload_gemms"] = workload_gemms(args.reps)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
