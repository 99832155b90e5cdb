"""The C ABI used from plain C: tests/c/abi_host.c is compiled with gcc
against include/ccl.h, linked with libccl.so and run (host-only calls, no
GPU). Its results must equal the Python binding's, which are pinned to the
oracle elsewhere."""
import os
import shutil
import subprocess

import pytest

from paper_2606_11718_amd import ccl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_11718_amd")


@pytest.fixture(scope="module")
def abi_output(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    ccl.library()                                   # the library is built
    exe = str(tmp_path_factory.mktemp("abi") / "abi_host")
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_host.c"), "-o", exe, "-L", PKG, "-lccl",
           f"-Wl,-rpath,{PKG}", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, HIP_VISIBLE_DEVICES="")   # host-only calls
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    return {ln.split()[0] + ("_" + ln.split()[1] if ln.startswith("remote") else ""): ln.split()[1:]
            for ln in r.stdout.splitlines()}


def test_plan_and_layout(abi_output):
    assert abi_output["grid"] == ["2", "4"]
    p = ccl.ccl_plan(8192, 28672, 8192, 8, 2, 4096)
    lay = ccl.ccl_plan_layout(p, ccl.CCL_B)
    assert list(map(int, abi_output["layout_b"])) == [lay.block_rows, lay.block_cols,
                                                      lay.strip_stride_bytes, lay.total_bytes]


def test_remote_bytes(abi_output):
    p = ccl.ccl_plan(8192, 28672, 8192, 8, 2, 4096)
    for pl in range(3):
        vals = abi_output[f"remote_{pl}"]
        ref = ccl.ccl_remote_bytes(p, pl, 0)
        assert list(map(int, vals[1:4])) == ref["remote"]
        assert int(vals[5]) == ref["floor"]
        assert int(vals[7]) == sum(ref["remote"])       # per-chiplet values add up


def test_l2_model(abi_output):
    p = ccl.ccl_plan_typed(256, 512, 256, 4, 2, 4096, ccl.CCL_DT_FP8_E4M3, ccl.CCL_DT_FP32)
    ref = ccl.ccl_remote_bytes_l2(p, ccl.CCL_PLACE_RR,
                                  ccl.CCL_TRAFFIC_A_TRANS | ccl.CCL_TRAFFIC_C_READ,
                                  l2_bytes=8 * 16 * 128, slots=2, k_step=128, traversal=1)
    assert list(map(int, abi_output["l2"])) == ref["accesses"] + ref["misses"] + ref["remote"]


def test_error_paths(abi_output):
    assert abi_output["err_plan"] == ["CCL_ERR_UNALIGNED_PARTITION", "1"]
    assert abi_output["err_null"] == ["CCL_ERR_INVALID_ARG"]
    assert abi_output["err_gemm"] == ["CCL_ERR_INVALID_ARG"]
    assert "ok" in abi_output


def test_splitk_workspace_query(abi_output):
    p = ccl.ccl_plan(768, 2048, 4096, 8, 1, 4096)
    assert list(map(int, abi_output["splitk"])) == list(ccl.ccl_gemm_splitk_workspace(p, 0))
