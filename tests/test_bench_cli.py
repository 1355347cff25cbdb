"""bench.py's contract where it does not need a GPU: more than one GPU is
refused with a message, a host without a GPU is refused cleanly, and the
cpu_baseline leg (the float64 oracle timed on a bounded sample) returns the
fields the JSON line carries."""
import os
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-GPU path")
def test_no_gpu_is_refused_cleanly():
    r = _run("--steps", "1", "--warmup", "0", "--no-cpu-baseline")
    assert r.returncode == 2
    assert "needs a GPU" in r.stderr
    assert r.stdout == ""


def test_cpu_baseline_fields():
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    w = workloads.make_workload("tiny")
    rec = bench.cpu_baseline(w, budget_s=0.5, max_rows=128)
    assert rec["kind"] == "oracle" and rec["unit"] == "scored tokens/s"
    assert rec["value"] > 0 and rec["cores"] >= 1
    assert "eligible rows" in rec["sample"]
