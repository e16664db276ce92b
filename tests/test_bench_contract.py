"""The benchmark's contract, checked on the CPU."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_dense_counters_describe_the_current_kernel():
    # The hardware-counter figures the bench line reports (VALU instructions per
    # evaluation, HBM bytes per launch) were taken on one version of the dense
    # kernel and its launch plan; they must be re-taken whenever that code changes.
    assert bench.dense_code_hash() == bench.DENSE_COUNTERS["dense_code_sha256_16"]
    src = os.path.join(ROOT, bench.DENSE_COUNTERS["source"])
    with open(src) as f:
        assert bench.DENSE_COUNTERS["dense_code_sha256_16"] in f.read()


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
