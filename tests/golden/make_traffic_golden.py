"""Write traffic_golden.json: the oracle's remote-byte records for every
workload GEMM, grid and page size (calls only oracle/ and the workload list).

Run from the repository root:  python tests/golden/make_traffic_golden.py
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402
from oracle import plan as PL, traffic as T  # noqa: E402


def main():
    out = []
    for wl in W.WORKLOADS.values():
        for g in wl.gemms:
            grids = [PL.auto_grid_rows(g.M, g.N, g.K, g.chiplets) if gr == 0 else gr for gr in g.grids]
            for gr, req in zip(grids, g.grids):
                gc = g.chiplets // gr
                for P in g.pages:
                    for pl in T.PLACEMENTS:
                        t0 = time.time()
                        rec = T.remote_bytes(g.M, g.N, g.K, gr, gc, P, pl, g.a_trans, g.b_trans)
                        rec.update(gemm=g.name, M=g.M, N=g.N, K=g.K, chiplets=g.chiplets,
                                   grid_rows_requested=req, grid_rows=gr, page=P, placement=pl,
                                   trans_a=g.a_trans, trans_b=g.b_trans)
                        out.append(rec)
                        print(f"{g.name} {gr}x{gc} P={P} {pl}: {T.total_remote(rec)} "
                              f"({time.time() - t0:.1f}s)", flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "traffic_golden.json")
    with open(path, "w") as f:
        json.dump({"_about": "oracle remote-byte records; written by make_traffic_golden.py",
                   "records": out}, f, indent=0)


if __name__ == "__main__":
    main()
