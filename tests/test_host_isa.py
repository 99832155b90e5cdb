"""Checks on the gfx950 assembly of the GEMM kernels, built here from source
(no GPU needed).

The 256x256 bf16 and fp8 kernels issue a wave's direct-to-LDS loads of one
operand in one step as a run that shares one M0 write: the first load of a
run sets M0 to the run's LDS destination, and load i of the run reaches LDS
1024 i bytes further through its instruction offset. That is correct only if
the compiler places no other M0 write inside a run and keeps the run's loads
in order. This test compiles gemm.hip to assembly and walks both kernels:
after every M0 write, the direct-to-LDS loads up to the next M0 write must
carry the instruction offsets 0, 1024, 2048, ... in that order. It also
checks that no register spill code sits inside their K loops.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_11718_amd import build as B

A2 = "_ZN3ccl12_GLOBAL__N_114gemm_a2_kernelENS0_10GemmParamsE"
FP8P = "_ZN3ccl12_GLOBAL__N_116gemm_fp8p_kernelENS0_10GemmParamsE"
# kernel: (lengths of its load runs, MFMAs of one iteration of its main loop)
KERNELS = {A2: ({2, 4}, 384), FP8P: ({4}, 192)}


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "gemm.s"
    src = os.path.join(B.CSRC, "kernels", "gemm.hip")
    cmd = [B.HIPCC] + B.HIP_FLAGS + ["-x", "hip", "--cuda-device-only", "-S", src, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return out.read_text()


def _body(asm_text: str, name: str) -> list:
    i = asm_text.index(name + ":")
    j = asm_text.index(".Lfunc_end", i)
    return [ln.strip() for ln in asm_text[i:j].splitlines()]


def _lds_offset(line: str) -> int:
    m = re.search(r"\boffset:(0x[0-9a-fA-F]+|\d+)", line)
    return int(m.group(1), 0) if m else 0


@pytest.mark.parametrize("kernel", list(KERNELS))
def test_load_runs_share_one_m0_write(asm, kernel):
    body = _body(asm, kernel)
    runs, run = [], None
    for ln in body:
        if re.match(r"s_\w+\s+m0\b", ln):
            if run is not None:
                runs.append(run)
            run = []
            continue
        if ln.startswith("buffer_load_dwordx4") and ln.endswith(" lds"):
            assert run is not None, f"direct-to-LDS load before any M0 write: {ln}"
            run.append(_lds_offset(ln))
    if run is not None:
        runs.append(run)
    assert len(runs) > 10, "expected the unrolled K loop's load runs"
    lengths = set()
    for r in runs:
        assert r == [1024 * i for i in range(len(r))], f"load run with offsets {r}"
        lengths.add(len(r))
    # bf16: A runs of 4 loads (one 64-K pair per wave) and B runs of 2 (one
    # 32-K stage); fp8: 4 loads per operand and 128-K stage
    assert lengths - {0} == KERNELS[kernel][0], lengths


@pytest.mark.parametrize("kernel", list(KERNELS))
def test_k_loop_has_no_spill_code(asm, kernel):
    body = _body(asm, kernel)
    labels = {m.group(1): n for n, ln in enumerate(body) if (m := re.match(r"^(\.LBB\S+):", ln))}
    mfmas = KERNELS[kernel][1]
    for n, ln in enumerate(body):
        m = re.search(r"s_cbranch_\w+\s+(\.LBB\S+)", ln)
        if m and labels.get(m.group(1), n) < n:
            loop = body[labels[m.group(1)]:n + 1]
            if sum(x.startswith("v_mfma") for x in loop) == mfmas:
                spills = [x for x in loop if x.startswith("scratch_") or re.match(r"v_(read|write)lane_b32", x)]
                assert not spills, spills[:4]
                return
    pytest.fail("main K loop not found")
