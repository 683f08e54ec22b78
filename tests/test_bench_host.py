"""Host-side checks of bench.py (no GPU): the one-GPU contract and the
algorithmic work it divides by the measured times."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synthetic as sy  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_algorithmic_work_single_sequence_workload():
    # batch 1, block 16, vocab 151936 in bf16, top-4, 65 tree rows over 4096
    # context keys, 8 KV heads and 32 query heads of dimension 128
    w = sy.workload(2)
    ctx = np.array([4096])
    n = np.array([65])
    depth = np.zeros((1, 65), np.int64)
    depth[0, 1:] = 1  # a star: the root and 64 children
    got = bench.algorithmic_work(w, ctx, n, depth)
    assert got["topk_bytes"] == 16 * 151936 * 2 + 16 * (8 * 4 + 4)          # rows, ids/logprob/lse
    assert got["argmax_bytes"] == 65 * 151936 * 2                           # one target row per node
    assert got["attn_bytes_per_layer"] == (8 * (4096 + 65) * 128 * 2 * 2      # K and V read once
                                           + 65 * 32 * 128 * 2 * 2)         # Q read, O written
    # every query row sees the context, its ancestors and itself: 4096 + depth + 1 keys,
    # two products of 2 d flops per key
    keys = 4096 * 65 + (1 + 64 * 2)
    assert got["attn_flops_per_layer"] == 32 * 4 * 128 * keys
