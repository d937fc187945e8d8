"""Host-side logic of bench.py (no GPU): the one-GPU guard and the
algorithmic byte counts its roofline figures divide by."""
import os
import subprocess
import sys

import bench
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_algorithmic_bytes_stage1():
    # sequence layout: u, delta (4 x 192 x 3136 fp32 each), B, C (4 x 16 x 3136),
    # y written once, and A, D, dt_bias
    s = workloads.STAGE1
    K, Dc, L, N = 4, 192, 3136, 16
    want_seq = (2 * K * Dc * L + 2 * K * N * L) * 4 + K * Dc * L * 4 + (K * Dc * N + 2 * K * Dc) * 4
    assert bench.seq_bytes(s, 1) == want_seq == 30562304
    # 2-D layout: x read once instead of u, the merged y written once
    want_2d = (Dc * L + K * Dc * L + 2 * K * N * L) * 4 + Dc * L * 4 + (K * Dc * N + 2 * K * Dc) * 4
    assert bench.ss2d_bytes(s, 1) == want_2d == 16111616
    # bf16 streams halve the streamed bytes, not the fp32 parameters
    b16 = bench.seq_bytes(workloads.BATCHED_BF16, 128, 2, 2)
    assert b16 == 128 * (2 * K * Dc * L + 2 * K * N * L) * 2 + 128 * K * Dc * L * 2 + \
        (K * Dc * N + 2 * K * Dc) * 4
