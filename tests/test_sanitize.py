"""The host code of the library (batch validation, planner, work accounting,
latency model, chunk selector: hb_plan.cpp and hb_predict.cpp, which make no
HIP call) built with AddressSanitizer and UndefinedBehaviorSanitizer and run
over seeded random batches, valid and malformed: no report, every sanitizer
finding is fatal."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2503_22562_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_under_address_and_undefined_behavior_sanitizers(tmp_path):
    exe = str(tmp_path / "sanitize_driver")
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    cmd = ["g++", "-O1", "-g", "-std=c++17", *san, f"-I{CSRC}", f"-I{os.path.join(ROOT, 'include')}",
           os.path.join(ROOT, "tests", "sanitize_driver.cpp"), os.path.join(CSRC, "hb_plan.cpp"),
           os.path.join(CSRC, "hb_predict.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, f"exit {r.returncode}\n{r.stdout}\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    print(r.stdout)
