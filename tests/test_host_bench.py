"""Host-side checks of bench.py (no GPU): the multi-GPU refusal, the remote-byte
report against the oracle's stored values, and the source hash that ties
the committed counter passes to the GEMM code they were taken on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

GOLDEN = os.path.join(ROOT, "tests", "golden", "traffic_golden.json")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_remote_report_matches_the_oracle_values():
    """Every 4 KB row of the report for the tiny configuration equals the
    totals the oracle wrote into the golden file."""
    rep = bench.remote_report()
    gold = json.load(open(GOLDEN))["records"]
    want = {}
    for g in gold:
        if g["gemm"] == "tiny" and g["page"] == 4096 and not g["trans_a"] and not g["trans_b"]:
            want[g["placement"]] = (sum(g["remote"]), g["floor"], sum(g["accessed"]))
    rows = [r for r in rep["rows"] if r["gemm"] == "tiny" and r["page"] == 4096]
    assert rows and set(want) == {"rr", "coarse", "ccl"}
    for r in rows:
        for pl in ("rr", "coarse", "ccl"):
            assert r[pl] == want[pl][0], pl
        assert r["floor"] == want["ccl"][1]
        assert r["accessed"] == want["ccl"][2]
        assert r["excess_ccl"] == 0


def test_kernel_hash_ignores_comments_and_layout(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("int f(int x) {\n  return x + 1;  // one\n}\n")
    b.write_text("/* header */\nint f(int x)\n{ return x + 1; }\n")
    c.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert bench.kernel_hash((str(a),)) == bench.kernel_hash((str(b),))
    assert bench.kernel_hash((str(a),)) != bench.kernel_hash((str(c),))


def test_committed_traffic_is_dropped_when_the_code_differs(tmp_path, monkeypatch):
    t = tmp_path / "traffic.json"
    t.write_text(json.dumps({"kernel_hash": "0" * 16, "hbm_bytes_per_launch": 123}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(t))
    assert bench.measured_traffic() is None
    t.write_text(json.dumps({"kernel_hash": bench.kernel_hash(), "hbm_bytes_per_launch": 123}))
    assert bench.measured_traffic() == 123


@pytest.mark.parametrize("src", bench.GEMM_SRCS)
def test_hashed_sources_exist(src):
    assert os.path.exists(src)


def test_tensor_parallel_shards_are_one_gpus_share_of_the_llama_ffn():
    """The workload leg's 8-way tensor-parallel shards: the up projection by
    output columns, the down projection by K; both plan (automatic grid) on
    whole 256x256 tiles of the 8 XCD partitions."""
    from paper_2606_11718_amd import ccl
    shapes = {name: (M, N, K) for name, M, N, K in bench.TP8_SHARDS}
    assert shapes == {"llama_up_tp8_shard": (8192, 3584, 8192),
                      "llama_down_tp8_shard": (8192, 8192, 3584)}
    for M, N, K in shapes.values():
        p = ccl.ccl_plan(M, N, K, 8, 0, 4096)
        tm, tn, wgs = ccl.ccl_debug_gemm_config(p)
        gr, gc = ccl.ccl_plan_grid(p)
        assert (tm, tn) == (256, 256) and gr * gc == 8
        assert wgs == 8 * (M // gr // 256) * (N // gc // 256)     # one partition per XCD
