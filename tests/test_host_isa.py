"""Checks on the gfx950 assembly of the GEMM kernels, built here from source
(no GPU needed).

The 256x256 bf16 kernel issues a wave's direct-to-LDS loads of one operand
in one step as a run that shares one M0 write: the first load of a run sets
M0 to the run's LDS destination, and load i of the run reaches LDS 1024 i
bytes further through its instruction offset. That is correct only if the
compiler places no other M0 write inside a run and keeps the run's loads in
order. This test compiles gemm.hip to assembly and walks gemm_a2_kernel:
after every M0 write, the direct-to-LDS loads up to the next M0 write must
carry the instruction offsets 0, 1024, 2048, ... in that order. It also
checks that the kernel spills no registers.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_11718_amd import build as B

KERNEL = "_ZN3ccl12_GLOBAL__N_114gemm_a2_kernelENS0_10GemmParamsE"


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


def test_a2_load_runs_share_one_m0_write(asm):
    body = _body(asm, KERNEL)
    runs, run = [], None
    for ln in body:
        if re.match(r"s_mov_b32\s+m0\b", ln) or re.match(r"s_\w+\s+m0\b", ln):
            if run is not None:
                runs.append(run)
            run = []
            continue
        if ln.startswith("buffer_load_dwordx4") and ln.endswith(" lds"):
            assert run is not None, f"direct-to-LDS load before any M0 write: {ln}"
            run.append(_lds_offset(ln))
    if run is not None:
        runs.append(run)
    assert len(runs) > 50, "expected the unrolled K loop's load runs"
    lengths = set()
    for r in runs:
        assert r == [1024 * i for i in range(len(r))], f"load run with offsets {r}"
        lengths.add(len(r))
    # A runs of 4 loads (one 64-K pair per wave) and B runs of 2 (one 32-K stage)
    assert lengths <= {0, 2, 4} and {2, 4} <= lengths, lengths


def test_a2_kernel_spills_nothing(asm):
    k = asm.index(".name:           " + KERNEL)
    end = asm.find("\n  - .", k)
    seg = asm[k:end if end > 0 else len(asm)]
    spills = {key: int(v) for key, v in re.findall(r"\.(sgpr_spill_count|vgpr_spill_count):\s+(\d+)", seg)}
    assert spills == {"sgpr_spill_count": 0, "vgpr_spill_count": 0}, spills
