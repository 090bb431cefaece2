"""bench.py's contract, on the CPU: one GPU only, and the algorithmic bytes and flops behind its
roofline fractions, restated here for the Llama-3-8B-shaped configuration by hand."""
import os
import subprocess
import sys

import bench
from synth import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_algorithmic_figures_at_the_llama3_8b_shape():
    # 32 layers, Patch layers {0, 8, 16, 24}, T = 8192, D = w = 1024 (g = 1), d_model = 4096,
    # rank 128 everywhere, offsets on the Reuse layers, aligner hidden width 4096, bf16 (2 bytes).
    wl = W.LLAMA3_8B
    alg = bench.algorithmic(wl)
    T, D, d, r, h, eb = 8192, 1024, 4096, 128, 4096, 2
    n_reuse, n_patch = 28, 4
    assert alg["kv_bytes"] == 32 * 2 * T * D * eb
    # Reuse decode per layer and branch: codes, basis and offset read once, the cache written once
    assert alg["reuse_decode"][0] == n_reuse * 2 * (T * r + D * r + D + T * D) * eb
    assert alg["reuse_decode"][1] == n_reuse * 2 * 2 * T * r * D
    # encode: inputs read once, basis and offset once, codes written once; H codes on Patch layers
    assert alg["encode"][0] == (n_reuse * 2 * (T * D + r * D + D + T * r)
                                + n_patch * (T * d + r * d + T * r)) * eb
    # Patch from the codes: act = SiLU(Z_H W1^T + b1) written once, read once by the folded
    # product act W_fold^T + c, whose K and V outputs are written once
    act_b = n_patch * (T * r + h * r + h + T * h) * eb
    gemm_b = n_patch * (T * h + 2 * D * h + 2 * D + 2 * T * D) * eb
    assert alg["patch"] == (act_b + gemm_b, n_patch * (2 * T * r * h + 2 * T * h * 2 * D))
    assert alg["patch"][1] == 584_115_552_256
