"""Register budgets of the GEMM, elementwise and probe kernels (CPU, hipcc only): no
instantiation spills VGPRs. A spill in an 8-wave GEMM tile lands in its K loop
(scratch traffic on every stage); the residual-epilogue instantiations once
spilled 40-103 registers that way."""
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc") and shutil.which("hipcc") is None, reason="no hipcc")
@pytest.mark.parametrize("src", ["k_gemm.hip", "k_elementwise.hip", "k_probe.hip"])
def test_no_vgpr_spills(src, tmp_path):
    from paper_2503_22562_amd import build as B
    cmd = [B.HIPCC, *B.COMMON, *B.HIP_FLAGS, *B.EXTRA_FLAGS.get(src, []), "--cuda-device-only",
           "-Rpass-analysis=kernel-resource-usage", "-c", os.path.join(B.CSRC, src), "-o", str(tmp_path / "k.o")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    names = re.findall(r"Function Name: (\S+)", r.stderr)
    spills = [int(v) for v in re.findall(r"VGPRs Spill: (\d+)", r.stderr)]
    assert names and len(names) == len(spills)
    bad = [(n, s) for n, s in zip(names, spills) if s]
    assert not bad, bad
