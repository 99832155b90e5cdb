"""Host C++ of the library under AddressSanitizer and UndefinedBehaviorSanitizer.

The real sources of the C-ABI layer and the host model (ccl_api.cpp,
host/plan.cpp, host/l2sim.cpp) are compiled with g++ -fsanitize=address,
undefined, against a test double of the few HIP runtime calls that layer
makes (tests/c/sanitize/hip/hip_runtime.h: one gfx950 device) and recording
stubs in place of the kernel launchers. A plain-C driver then runs plans,
layouts, both traffic models (the finite-L2 one with several host threads),
one plan from several threads, the split-K workspace query, the workgroup
map and the argument checks of every device call. Any sanitizer report
fails the run; every value must equal the regular library's.
"""
import os
import shutil
import subprocess

import pytest

from paper_2606_11718_amd import ccl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_11718_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "c", "sanitize")
FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         "-g", "-O1"]

SHAPES = [(256, 512, 256, 4, 2, 4096, 0, 0), (4096, 1536, 2048, 8, 2, 4096, 0, 0),
          (768, 2048, 4096, 8, 0, 4096, 0, 0), (4096, 768, 2048, 8, 0, 4096, 0, 0),
          (8192, 28672, 8192, 8, 2, 4096, 0, 0), (8192, 8192, 28672, 8, 4, 65536, 0, 0),
          (8192, 28672, 8192, 8, 8, 2097152, 0, 0), (1024, 768, 1024, 8, 8, 4096, 1, 2),
          (384, 768, 384, 3, 1, 4096, 2, 2)]


@pytest.fixture(scope="module")
def run(tmp_path_factory):
    for tool in ("g++", "gcc"):
        if shutil.which(tool) is None:
            pytest.skip(f"{tool} not available")
    d = tmp_path_factory.mktemp("sanitize")
    inc = ["-I", SAN, "-I", CSRC]
    objs = []
    for src in (os.path.join(CSRC, "host", "plan.cpp"), os.path.join(CSRC, "host", "l2sim.cpp"),
                os.path.join(CSRC, "ccl_api.cpp"), os.path.join(SAN, "launch_stubs.cpp")):
        obj = str(d / (os.path.basename(src) + ".o"))
        cmd = ["g++", "-std=c++17", "-pthread", "-Wall"] + FLAGS + inc + ["-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        objs.append(obj)
    drv = str(d / "driver.o")
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror"] + FLAGS +
                       ["-I", os.path.join(ROOT, "include"), "-c", os.path.join(SAN, "driver.c"),
                        "-o", drv], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    exe = str(d / "san")
    r = subprocess.run(["g++", "-pthread"] + FLAGS + objs + [drv, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
    assert "Sanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-6000:]
    recs = {}
    for ln in r.stdout.splitlines():
        kind, *rest = ln.split()
        recs.setdefault(kind, []).append(rest)
    return recs


def _plans():
    return [ccl.ccl_plan_typed(M, N, K, G, Gr, P, ab, c) for M, N, K, G, Gr, P, ab, c in SHAPES]


def test_no_mismatch_and_every_valid_device_call_reached_its_launcher(run):
    assert run["failures"] == [["0"]]
    assert "MISMATCH" not in run
    assert run["launches"] == [["11"]]


def test_plans_layouts_and_traffic_equal_the_library(run):
    plans = _plans()
    for i, g, c in ((int(a), int(b), int(c)) for a, b, c in run["grid"]):
        assert ccl.ccl_plan_grid(plans[i]) == (g, c)
    for rec in run["layout"]:
        i, op, *vals = map(int, rec)
        lay = ccl.ccl_plan_layout(plans[i], op)
        assert vals == [lay.block_rows, lay.block_cols, lay.strip_stride_bytes, lay.total_bytes]
    assert len(run["traffic"]) == len(SHAPES) * 24
    for rec in run["traffic"]:
        i, pl, flags, *vals = map(int, rec)
        ref = ccl.ccl_remote_bytes(plans[i], pl, flags)
        assert vals[0:3] == ref["accessed"] and vals[3:6] == ref["remote"]
        assert vals[6] == ref["floor"] and vals[7] == sum(ref["remote"])


def test_workgroup_map_equals_the_library(run):
    plans = _plans()
    assert len(run["tilemap"]) == len(SHAPES) - 1          # the fp32-operand plan has no GEMM
    for rec in run["tilemap"]:
        i, rows, cols, wgs, h = map(int, rec)
        assert ccl.ccl_debug_gemm_config(plans[i]) == (rows, cols, wgs)
        want = 0
        for wg in range(wgs):
            xcd, tm, tn = ccl.ccl_debug_tile_of_wg(plans[i], wg)
            want = (want * 1000003 + xcd + 8 * (tm + 1) + 8 * 65536 * (tn + 1)) % (1 << 64)
        assert h == want, i


def test_l2_model_and_splitk_query_equal_the_library(run):
    plans = _plans()
    for rec in run["l2"]:
        i, trav, threads, *vals = map(int, rec)
        ref = ccl.ccl_remote_bytes_l2(plans[i], ccl.CCL_PLACE_RR, ccl.CCL_TRAFFIC_C_READ,
                                      l2_bytes=64 * 16 * 128, ways=16, line_bytes=128, slots=4,
                                      k_step=64, traversal=trav, threads=threads, group_rows=2)
        assert vals == ref["accesses"] + ref["misses"] + ref["remote"]
    for req, splits, ws in (map(int, r) for r in run["splitk"]):
        assert ccl.ccl_gemm_splitk_workspace(plans[2], req) == (splits, ws)
    sums = {tuple(r) for r in run["threads"]}
    assert len(sums) == 1
