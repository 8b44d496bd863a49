"""Host checks of bench.py's measurement bookkeeping (no GPU): the committed
counter summary belongs to the committed softmax sources, so the benchmark's
roofline.traffic is reported rather than null, and the --gpus contract for
more than one GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_committed_counters_match_the_softmax_sources():
    # The counter summary records a hash of softmax.hip and kf_device.hpp;
    # a kernel change without fresh counter passes makes traffic null.
    traffic = bench.measured_traffic()
    assert traffic is not None, "profiles/ counters predate the current softmax sources"
    algorithmic = 1 * 8 * 4096 * 4096 * 2 * 2
    assert 0.99 <= traffic / algorithmic <= 1.05


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr), r.stdout + r.stderr
