"""bench.py without a GPU: the multi-GPU refusal and the helpers that label
and summarise its measurements."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_percentile_and_spread():
    xs = [5.0, 1.0, 3.0, 2.0, 4.0]
    assert bench.percentile(xs, 0) == 1.0 and bench.percentile(xs, 100) == 5.0
    assert bench.percentile(xs, 50) == 3.0
    assert bench.percentile(xs, 10) == pytest.approx(1.4)
    assert bench.percentile([7.0], 90) == 7.0
    s = bench.spread(xs)
    assert s == {"median": 3.0, "p10": 1.4, "p90": 4.6, "n": 5}


def test_labels_follow_the_launch_rules():
    # span of a bulk launch: power of two at or above a quarter of the tile, 2..32 rows of 1 KiB
    assert bench.bulk_span_rows(131072) == 32      # LLaMA-7B tiles
    assert bench.bulk_span_rows(53248) == 16       # LLaMA-30B quarter
    assert bench.bulk_span_rows(32768) == 8        # GQA
    assert bench.bulk_span_rows(8192) == 2         # tiny
    assert bench.bulk_span_rows(1 << 30) == 32
    assert bench.inline_launch(4096, 4096) == (2, 512)
    assert bench.inline_launch(65536, 100) == (2, 512)
    assert bench.inline_launch(65537, 100) == (1, 256)


def test_stage_bytes_counts_read_and_write():
    class Shape:
        num_layers = 32
    assert bench.stage_bytes(512, Shape, 131072) == 8589934592
