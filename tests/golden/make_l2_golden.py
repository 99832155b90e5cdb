"""Write l2_golden.json: the oracle's finite-L2 traffic records for the Qwen3
workload GEMMs (calls only oracle/ and the workload list).

Run from the repository root:  python tests/golden/make_l2_golden.py
"""
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402
from oracle import l2sim as L, plan as PL  # noqa: E402

MIB = 1 << 20
# (chiplets, l2 bytes per chiplet, resident tiles per chiplet):
#   MI355X-like: 8 XCDs of 32 CUs with 4 MB L2 each, and a smaller L2;
#   the paper's MI300X-like setting: 4 domains of 76 CUs with 8 MB L2 each.
SETTINGS = [(8, 4 * MIB, 32), (8, 1 * MIB, 32), (4, 8 * MIB, 76)]


def _cases():
    for wl in ("qwen_fwd", "qwen_bwd"):
        for g in W.WORKLOADS[wl].gemms:
            for chiplets, l2, slots in SETTINGS:
                gr = PL.auto_grid_rows(g.M, g.N, g.K, chiplets)
                if gr == 0:
                    continue
                for pl in ("rr", "coarse", "ccl"):
                    for trav in ("row", "col"):
                        yield dict(gemm=g.name, M=g.M, N=g.N, K=g.K, chiplets=chiplets, grid_rows=gr,
                                   page=4096, placement=pl, trans_a=g.a_trans, trans_b=g.b_trans,
                                   l2_bytes=l2, ways=16, line=128, slots=slots, k_step=64,
                                   traversal=trav)


def _run(c):
    t0 = time.time()
    rec = L.simulate(c["M"], c["N"], c["K"], c["grid_rows"], c["chiplets"] // c["grid_rows"], c["page"],
                     c["placement"], c["trans_a"], c["trans_b"], l2_bytes=c["l2_bytes"],
                     ways=c["ways"], line=c["line"], slots=c["slots"], k_step=c["k_step"],
                     traversal=c["traversal"])
    rec.update(c)
    return rec, time.time() - t0


def main():
    out = []
    with ProcessPoolExecutor(max_workers=8) as ex:
        for rec, dt in ex.map(_run, list(_cases())):
            out.append(rec)
            print(f"{rec['gemm']} G={rec['chiplets']} L2={rec['l2_bytes'] >> 20}MB {rec['placement']} "
                  f"{rec['traversal']}: {L.total_remote(rec)} ({dt:.1f}s)", flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "l2_golden.json")
    with open(path, "w") as f:
        json.dump({"_about": "oracle finite-L2 traffic records; written by make_l2_golden.py",
                   "records": out}, f, indent=0)


if __name__ == "__main__":
    main()
