"""Host checks of the benchmark's accounting (no GPU): the work and byte counts it
divides by, against the workload's closed forms and the figures of the
algorithmic-work table for the Qwen3-8B shape (K read 2.49 GB, V read 2.42 GB,
QK^T 1.28 TFLOP for one pass), and its refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_03928_amd import synth  # noqa: E402

CFG = synth.CONFIGS["qwen3-8b"]


def test_score_flops_is_one_pass_of_qk():
    n, R, N, d = CFG.n_inst, CFG.G * CFG.w, CFG.K + CFG.B, CFG.d
    assert bench.score_flops(CFG) == 2 * n * R * N * d
    assert abs(bench.score_flops(CFG) / 1e12 - 1.28) < 0.005


def test_round_bytes_components():
    n, K, B, d, e = CFG.n_inst, CFG.K, CFG.B, CFG.d, CFG.elem_bytes
    N = K + B
    k_read, v_read = n * N * d * e, n * K * d * e
    assert abs(k_read / 1e9 - 2.49) < 0.005 and abs(v_read / 1e9 - 2.42) < 0.005
    ab = bench.algorithmic_bytes(CFG, moved_rows=0, reads_values=True, layout="stable")
    window = n * CFG.G * CFG.w * d * e
    assert ab["score"] == k_read + v_read + window + n * 2 * K * 4
    # without V (carried value scores) the score reads K, the window and its arrays
    ab2 = bench.algorithmic_bytes(CFG, moved_rows=0, reads_values=False, layout="stable")
    assert ab["score"] - ab2["score"] == v_read
    # every moved row is read and written for K and V
    ab3 = bench.algorithmic_bytes(CFG, moved_rows=1000, reads_values=True, layout="stable")
    assert ab3["compact_decode"] - ab["compact_decode"] == 1000 * 2 * d * e


def test_compaction_alone_bytes_under_the_map():
    n, K, B, d, e = CFG.n_inst, CFG.K, CFG.B, CFG.d, CFG.elem_bytes
    # survivor map and order map read, new map written, B rows of K and V read and written
    assert bench.compact_only_bytes(CFG, n * B, "map") == n * (12 * K + 4 * B * d * e)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr
