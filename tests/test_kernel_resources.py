"""Compile-time resource checks of the staged multiply (no GPU needed).

The staged multiply is written to keep its whole work-item state in
registers: a spill to scratch memory there is written back once per work item
(about 1.3 GB per 32K launch when the item descriptor was spilled) and each
reload waits for every load in flight.  These checks compile the kernel for
gfx950 and read the compiler's resource report."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32259_amd", "csrc")
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _resources(src, kernel, tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "--cuda-device-only", "-c",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           "-Rpass-analysis=kernel-resource-usage", os.path.join(CSRC, src),
           "-o", str(tmp_path / "k.o")]
    out = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert out.returncode == 0, out.stdout[-2000:]
    res, cur = {}, None
    for line in out.stdout.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", line)
        if m and cur and kernel in cur:
            res[m.group(1).strip()] = int(m.group(2))
    assert res, f"no resource report for {kernel}"
    return res


def test_staged_multiply_uses_no_scratch_and_fits_lds(tmp_path):
    # the common instantiation (no key norm); the key-norm one may spill a few
    # registers, stored once per launch
    r = _resources("staged.hip", "staged_gemm_kernelILb0", tmp_path)
    assert r["ScratchSize"] == 0, r
    assert r["VGPRs Spill"] == 0, r
    assert r["LDS Size"] <= 160 * 1024, r
    assert r["Occupancy"] >= 2, r   # two waves per SIMD: 8 waves in one workgroup per CU
