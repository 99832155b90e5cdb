"""CPU tests of the FFN GEMM sweep (paper_2606_11718_amd/sweep.py, Sec. IV-A
protocol): the 36 shapes, the per-placement minimum over grids and tile
traversals, the coarse/fine classification and the geometric means. The
library's values are compared with the oracle's models minimised the same
way, on small FFN shapes."""
import math

import pytest

import workloads as W
from oracle import l2sim as OL2
from oracle import plan as OP
from oracle import traffic as OT
from paper_2606_11718_amd import sweep

PLACE_ORACLE = {"rr_4k": ("rr", 4096), "rr_64k": ("rr", 65536), "rr_2m": ("rr", 2 << 20),
                "coarse": ("coarse", 4096), "ccl": ("ccl", 4096)}


def test_sweep_has_the_36_gemms():
    g = W.FFN_SWEEP
    assert len(g) == 36
    assert len({x.name for x in g}) == 36
    assert {x.tokens for x in g} == {4096, 8192, 16384}
    assert sum(x.pass_ == "fwd" for x in g) == 12
    # the workloads used elsewhere are sweep members with the same shape and storage
    for name in ("qwen_gate_up", "qwen_dW_down", "qwen_dH", "llama_up", "llama_down",
                 "llama_dW_up", "llama_dX"):
        _, wg = W.gemm_by_name(name)
        assert any((x.M, x.N, x.K, x.a_trans, x.b_trans) == (wg.M, wg.N, wg.K, wg.a_trans, wg.b_trans)
                   for x in g), name
    for x in g:                     # dX and dW of a layer share its dimensions
        if x.pass_ == "dX":
            assert x.b_trans == 1 and x.a_trans == 0
        if x.pass_ == "dW":
            assert x.a_trans == 1 and x.K == x.tokens


def _toy():
    out = []
    for T in (256, 512):
        for proj, din, dout in (("gate_up", 256, 512), ("down", 512, 256)):
            out.append(W.SweepGemm("toy", T, proj, "fwd", T, dout, din, 0, 0))
            out.append(W.SweepGemm("toy", T, proj, "dX", T, din, dout, 0, 1))
            out.append(W.SweepGemm("toy", T, proj, "dW", din, dout, T, 1, 0))
    return out


def _oracle_best(g, G, model, setting, e=(2, 2, 2)):
    best = {}
    for name, (pl, page) in PLACE_ORACLE.items():
        for gr in range(1, G + 1):
            if not OP.grid_valid(g.M, g.N, g.K, G, gr):
                continue
            for trav in (("row", "col") if model == "l2" else ("row",)):
                if model == "charge":
                    rb = OT.total_remote(OT.remote_bytes(g.M, g.N, g.K, gr, G // gr, page, pl,
                                                         g.a_trans, g.b_trans, e=e))
                else:
                    rb = OL2.total_remote(OL2.simulate(
                        g.M, g.N, g.K, gr, G // gr, page, pl, g.a_trans, g.b_trans,
                        l2_bytes=setting["l2_bytes"], slots=setting["slots"], ways=sweep.WAYS,
                        line=sweep.LINE, k_step=sweep.LINE // e[0], traversal=trav, e=e))
                if name not in best or rb < best[name]:
                    best[name] = rb
    return best


@pytest.mark.parametrize("model", ["charge", "l2"])
def test_best_configuration_matches_oracle(model):
    setting = dict(chiplets=4, l2_bytes=64 * 1024, slots=3)
    gemms = _toy()
    recs = sweep.evaluate(gemms, setting, model, workers=4)
    for g, r in zip(gemms, recs):
        want = _oracle_best(g, 4, model, setting)
        for name in PLACE_ORACLE:
            assert r[name]["remote_bytes"] == want[name], (g.name, name)
        assert r["coarse_optimal"] == (want["coarse"] <= want["ccl"])


@pytest.mark.parametrize("ab,c,e", [(1, 0, (1, 1, 2)), (2, 2, (4, 4, 4))])
def test_typed_best_configuration_matches_oracle(ab, c, e):
    """fp8 operands with a bf16 C, and fp32 throughout (Fig. 7 data types)."""
    setting = dict(chiplets=4, l2_bytes=64 * 1024, slots=3)
    gemms = _toy()[:6]
    recs = sweep.evaluate(gemms, setting, "l2", workers=4, ab_type=ab, c_type=c)
    for g, r in zip(gemms, recs):
        want = _oracle_best(g, 4, "l2", setting, e)
        for name in PLACE_ORACLE:
            assert r[name]["remote_bytes"] == want[name], (g.name, name)
        assert r["elem_bytes"] == list(e)


def test_gemm_without_aligned_grid_is_reported():
    g = W.SweepGemm("toy", 384, "down", "fwd", 384, 384, 256, 0, 0)     # 3 x 3 tiles, G = 4
    (r,) = sweep.evaluate([g], dict(chiplets=4, l2_bytes=0, slots=1), "charge", workers=1)
    assert r["no_aligned_grid"]
    assert sweep.summarize([r])["toy"]["gemms"] == 0


def test_summary_geomeans_and_counts():
    def rec(model, rr, coarse, ccl):
        r = {"model": model, "coarse_optimal": coarse <= ccl}
        for name, b in (("rr_4k", rr), ("rr_64k", rr), ("rr_2m", rr), ("coarse", coarse), ("ccl", ccl)):
            r[name] = {"remote_bytes": b}
        return r
    recs = [rec("m", 400, 100, 100), rec("m", 900, 300, 100), rec("m", 100, 200, 50)]
    s = sweep.summarize(recs)["m"]
    assert s["gemms"] == 3 and s["fine_optimal"] == 2
    assert math.isclose(s["rr_4k_over_ccl_gmean"], (4 * 9 * 2) ** (1 / 3))
    assert math.isclose(s["coarse_over_ccl_gmean"], (1 * 3 * 4) ** (1 / 3))
    assert math.isclose(s["coarse_over_ccl_gmean_fine_optimal"], (3 * 4) ** 0.5)
    assert s["rr_4k_over_ccl_max"] == 9


def test_ccl_never_loses_in_the_charge_model():
    """In the no-cache model CCL reaches the floor, so no placement beats it."""
    recs = sweep.evaluate([g for g in W.FFN_SWEEP if g.model == "qwen3_30b" and g.tokens == 4096],
                          "mi355x", "charge", workers=4)
    for r in recs:
        assert all(r[n]["remote_bytes"] >= r["ccl"]["remote_bytes"] for n in PLACE_ORACLE)
