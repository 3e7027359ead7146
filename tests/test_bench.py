"""Host-side checks of bench.py: it measures one GPU only, and its CPU-baseline leg
times the oracle on whole sequences of a workload (CPU only)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_worker_counts_rows():
    sys.path.insert(0, ROOT)
    import bench
    rows, secs = bench._cpu_baseline_worker(("tiny", 0, 0, 1))
    assert rows == 4 + 4 + 1          # k_max drafter rows and k_max + 1 target rows of one sequence
    assert secs > 0.0
