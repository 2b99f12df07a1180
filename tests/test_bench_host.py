"""Host logic of bench.py (no GPU): the one-GPU exit, the algorithmic byte counts behind `value` and `roofline`, and
the source-hash gate on the committed traffic figure."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout.strip() == ""


def test_apply_bytes_at_the_benchmark_shape():
    # 32 layers x {K,V} x 8 heads x 32768 rows of 2 x 256 bytes (read + written) and 64 coefficient bytes, plus the
    # fp32 bases once per unit: 16,777,216 x 576 + 512 x 32 x 128 x 4
    assert bench._apply_bytes(32, 8, 128, 32768, 32) == 16777216 * 576 + 512 * 32 * 128 * 4 == 9672065024
    # rank 0 moves the rows only
    assert bench._apply_bytes(32, 8, 128, 32768, 0) == 16777216 * 512


def test_fit_bytes_are_two_passes_over_both_caches():
    rows = 32 * 2 * 8 * 32768
    assert bench._fit_bytes(32, 8, 128, 32768, 32) == rows * (2 * 2 * 128 * 2 + 32 * 2)


def test_anchor_byte_counts():
    L, H, d, T, V, r = 32, 8, 128, 4096, 10, 32
    rows = L * 2 * H * T
    bases = V * L * 2 * H * r * d * 4
    assert bench._anchored_bytes(L, H, d, T, V, r) == rows * (2 * d * 2 + V * r * 2) + L * 2 * T * V * 4 * H + bases
    assert bench._weights_bytes(L, H, d, T, V, r) == rows * (d * 2 + V * r * 2) + L * 2 * T * V * 4 + bases


def test_traffic_is_reported_only_for_the_source_it_was_taken_on():
    with open(os.path.join(ROOT, "profiles", "kvc_apply_llama8b_32k_traffic.json")) as f:
        rec = json.load(f)
    assert bench._traffic(rec["source_hash"]) == rec["traffic_bytes_per_launch"]
    assert bench._traffic("0" * 16) is None
