"""The benchmark's command-line contract on the CPU: more than one GPU is
refused with a message and no work, and the calibrated-traffic lookup
returns nothing for a workload without a counter summary."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_lookup_without_a_summary():
    sys.path.insert(0, ROOT)
    import bench

    assert bench.digest_traffic("no-such-workload") is None
