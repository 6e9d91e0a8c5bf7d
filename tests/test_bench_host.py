"""Host-side logic of bench.py: the algorithmic byte counts behind the
reported GB/s and the one-GPU guard (no GPU needed)."""
import subprocess
import sys
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import inputs  # noqa: E402


def test_bytes_required_counts_prefixes_scales_and_vectors():
    # K = 256 (two groups), N = 512, levels {0, 2, 4, 8}: the first group all
    # skipped, the second group's rows at 2, 4 and 8 bits.
    K, N = 256, 512
    lm = np.zeros((1, K), np.uint8)
    lm[0, 128:160] = 1
    lm[0, 160:200] = 2
    lm[0, 200:256] = 3
    code = (32 * 2 + 40 * 4 + 56 * 8) * N // 8
    scales = 1 * N * 2                 # one active group, fp16 scales
    vectors = 2 * K + 4 * N             # fp16 x in, fp32 y out
    got = bench.bytes_required(lm, (0, 2, 4, 8), K, N, False)
    assert got.tolist() == [code + scales + vectors]
    assert bench.bytes_required(lm, (0, 2, 4, 8), K, N, True).tolist() == [code + scales + vectors + K]


def test_bytes_required_batch_reads_union_depth_once():
    K, N = 128, 256
    a = np.zeros((2, K), np.uint8)
    a[0, :64] = 3                       # token 0: first half at 8 bits
    a[1, 32:] = 1                       # token 1: the rest (and overlap) at 2 bits
    depth = np.maximum(np.array((0, 2, 4, 8))[a[0]], np.array((0, 2, 4, 8))[a[1]])
    want = int(depth.sum()) * N // 8 + 1 * N * 2 + 2 * (2 * K + 4 * N)
    assert bench.bytes_required_batch(a, (0, 2, 4, 8), K, N, False) == want
    # one token alone is the batch-1 count
    assert bench.bytes_required_batch(a[:1], (0, 2, 4, 8), K, N, False) == \
        int(bench.bytes_required(a[:1], (0, 2, 4, 8), K, N, False)[0])


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
