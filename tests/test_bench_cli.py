"""bench.py's command line on the CPU: more than one GPU is refused with a
message before anything touches a device, and the algorithmic work it
reports follows the closed forms of the layer."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_layer_work_closed_form():
    sys.path.insert(0, ROOT)
    import bench
    from hb_workloads import LLAMA3_8B
    reqs = [(512, 100), (1, 300), (1, 0)]
    fl, by = bench.layer_work(LLAMA3_8B, reqs)
    T = 514
    pairs = 512 * 100 + 512 * 513 / 2 + 300 + 1 + 1
    assert np.isclose(fl, 2 * T * 218103808 + 4 * 32 * 128 * pairs)
    kv_tok = 612 + 301 + 1
    assert np.isclose(by, 2 * 218103808 + 4 * 4096 + 2 * 2 * 8 * 128 * (kv_tok + T) + 2 * T * 4096 + 4 * T * 4096)
    # per-kernel flops add up to the layer's (the norms' 4TH aside), and the
    # per-kernel bytes partition the layer's algorithmic bytes exactly
    kw = bench.kernel_work(LLAMA3_8B, reqs)
    gemm_attn = sum(kw[k][0] for k in ("gemm_qkv", "attention", "gemm_o", "gemm_gate_up", "gemm_down"))
    assert np.isclose(gemm_attn, fl)
    assert np.isclose(sum(b for _, b in kw.values()), by)
    # attention moves the cached and new K/V once per (request, kv head), nothing else
    assert np.isclose(kw["attention"][1], 2 * 2 * 8 * 128 * kv_tok)
    # the layer's roofline time is the sum over kernels of max(F/peak, B/peak)
    want = sum(max(f / bench.PEAK_BF16, b / bench.PEAK_HBM) for f, b in kw.values())
    assert np.isclose(bench.roofline_time_s(kw), want)
    assert bench.roofline_time_s(kw) > max(fl / bench.PEAK_BF16, by / bench.PEAK_HBM)
