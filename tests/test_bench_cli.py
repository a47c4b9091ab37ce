"""The benchmark's command-line contract that holds without a GPU: one GPU
only, and the oracle's CPU baseline record."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = run_bench("--gpus", n)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_cpu_baseline_record():
    sys.path.insert(0, ROOT)
    import bench
    from workloads import config_shapes, make_inputs
    rec = bench.cpu_baseline(make_inputs(config_shapes(1)[0]), 0.2)
    assert rec["kind"] == "oracle" and rec["unit"] == "us/call"
    assert rec["value"] > 0 and rec["cores"] >= 1
    assert "full calls" in rec["sample"]
