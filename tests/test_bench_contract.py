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


class _Ev:
    """A stand-in for a timing event: a timestamp in ms."""

    def __init__(self, t):
        self.t = t

    def elapsed_time(self, other):
        return other.t - self.t


def test_consumer_span_and_phase_split_come_from_alternate_steps():
    # Even steps carry an event between the decode and Patch calls; the GPU idles 0.005 ms at it.
    # Encode 0.4, decode 0.3, Patch 0.5 ms every step.
    events, split = [], []
    t = 0.0
    for i in range(6):
        sp = i % 2 == 0
        gap = 0.005 if sp else 0.0
        e0 = _Ev(t)
        e1 = _Ev(t + 0.4)
        e2 = _Ev(t + 0.4 + 0.3)
        e3 = _Ev(t + 0.4 + 0.3 + gap + 0.5)
        events.append([e0, e1, e2, e3])
        split.append(sp)
        t += 2.0
    phase, consumer = bench.reduce_events(events, split)
    assert len(phase["encode"]) == 6
    assert len(phase["reuse_decode"]) == len(phase["patch"]) == len(consumer) == 3
    # the consumer span has no event gap in it; the phase split comes from the split steps only
    assert all(abs(c - 0.8) < 1e-12 for c in consumer)
    assert all(abs(x - 0.3) < 1e-12 for x in phase["reuse_decode"])
    assert all(abs(x - 0.505) < 1e-12 for x in phase["patch"])
    # one step (every step split): the consumer span comes from it
    phase1, consumer1 = bench.reduce_events(events[:1], [True])
    assert len(consumer1) == 1 and abs(consumer1[0] - 0.805) < 1e-12
