"""The benchmark's host-side contract, without a GPU: more than one GPU is
refused with a message, and the CPU-oracle baseline leg reports the fields
the JSON line carries."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_cpu_baseline_leg_on_a_tiny_sample():
    pytest.importorskip("threadpoolctl")
    sys.path.insert(0, ROOT)
    import bench
    from workloads import WORKLOADS
    cb = bench.cpu_baseline(WORKLOADS["single-1152"], rows=8, wrows=16)
    assert cb["kind"] == "oracle" and cb["unit"] == "TFLOP/s"
    assert cb["value"] > 0 and cb["cores"] >= 1
    assert "8 activation rows x 16 weight rows" in cb["sample"]
