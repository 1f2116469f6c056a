"""Host-side logic of bench.py, on the CPU: the algorithmic byte count of a
round and the single-GPU guard."""
from __future__ import annotations

import os
import subprocess
import sys

import bench
from paper_2608_02123_amd.synth import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_algorithmic_bytes_qwen4b_b16():
    # V = 151936, B = 16, r = 256, k = 8, R = 1, bf16, summed by hand:
    # W once per depth  16 * 256 * 151936 * 2 = 1,244,659,712
    # L_d               16 * 151936 * 2       =     4,861,952
    # frontier E rows   (1 + 15 * 8) * 256 * 2 =        61,952
    # h_d               16 * 256 * 4          =        16,384
    assert bench.algorithmic_bytes(CONFIGS["qwen4b_b16"]) == 1_249_600_000


def test_algorithmic_bytes_k_above_vocabulary():
    # k' = min(k, V): a 5-token vocabulary with k = 8 has frontiers of 5
    w = CONFIGS["qwen4b_b16"]
    small = type(w)("t", V=5, B=3, N=8, k=8, r=16, R=2, dtype="f32")
    expect = 3 * 16 * 5 * 4 + 2 * 3 * 5 * 4 + 2 * (1 + 2 * 5) * 16 * 4 + 2 * 3 * 16 * 4
    assert bench.algorithmic_bytes(small) == expect


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_w_once_bytes_qwen4b_b16():
    # W counted once per round (the on-chip floor), the rest as above:
    # 256 * 151936 * 2 = 77,791,232, + 4,861,952 + 61,952 + 16,384 = 82,731,520
    assert bench.algorithmic_bytes(CONFIGS["qwen4b_b16"], w_once=True) == 82_731_520


def test_spread_percentiles():
    sp = bench.spread([float(x) for x in range(1, 12)])  # 1 .. 11
    assert sp == {"median": 6.0, "p10": 2.0, "p90": 10.0, "rounds": 11}
    assert bench.spread([]) is None
