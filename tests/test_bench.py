"""bench.py host paths that need no GPU: the single-GPU guard and the CPU
oracle baseline it reports beside the GPU figures."""
import os
import subprocess
import sys

import bench
from dconv_workloads import WORKLOADS, make

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "one GPU" in (res.stdout + res.stderr)


def test_cpu_baseline_reports_the_oracle():
    w = WORKLOADS["single_64x64_m1_k3"]
    I, F = make(w)
    cb = bench.cpu_baseline([(w, I, F)], 2, min_seconds=0.0)
    assert cb["kind"] == "oracle" and cb["unit"] == "GFLOP/s"
    assert cb["value"] > 0 and cb["single_thread_value"] > 0
    assert cb["cores"] >= 1 and cb["affinity_cpus"] >= 1
    assert "repetitions" in cb["sample"]
