"""CPU checks of bench.py's byte accounting (the algorithmic bytes behind the roofline) against closed
forms for the Llama-3-8B-shaped workload, and of the JSON contract's refusal of more than one GPU."""

import os
import subprocess
import sys

import bench
from paper_2510_13223_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_partial_algorithmic_bytes_closed_form():
    w = workloads.make_config("llama3_8b", 0)
    B, Hq, Hkv = 64, 32, 8
    per_token = Hkv * 128 * 2 * 2  # K and V, bf16: the paper's 4096 B per token per layer
    assert per_token == 4096
    q_bytes = B * Hq * 128 * 2
    out_bytes = B * Hq * (128 + 1) * 4
    for part, blocks in ((0, 179), (1, 77)):
        total, kv = bench._partial_algorithmic_bytes(w, part)
        assert kv == B * blocks * 16 * per_token
        assert total == kv + q_bytes + B * blocks * 4 + B * 8 + out_bytes
    assert w.kv_bytes() == B * 4096 * per_token == 1 << 30


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
