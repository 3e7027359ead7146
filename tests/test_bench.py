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


def test_read_probe_library_checks_its_arguments():
    # the bench's bare-read probe: loads, exports its entry point, and rejects bad
    # arguments on the host before any launch (no GPU needed for these calls)
    import ctypes as C
    from paper_2508_15371_amd import build as B
    lib = C.CDLL(B.PROBE_LIB)
    f = lib.cmsd_probe_read_rows
    i64, vp = C.c_int64, C.c_void_p
    f.argtypes = [vp, i64, i64, vp, i64, i64, i64, C.c_int, C.c_int, vp, vp]
    f.restype = C.c_int
    fake = C.c_void_p(4096)
    assert f(fake, 4, 100, fake, 4, 100, 100, 96, 4, fake, None) == 1        # workgroup size
    assert f(fake, 4, 100, fake, 4, 100, 100, 256, 3, fake, None) == 1       # loads in flight
    assert f(fake, 4, 64, fake, 4, 100, 100, 256, 4, fake, None) == 1        # stride below the row
    assert f(None, 4, 100, fake, 0, 100, 100, 256, 4, fake, None) == 1       # rows without a base
    assert f(fake, 4, 100, fake, 4, 100, 100, 256, 4, None, None) == 1       # no sink
    assert f(fake, -1, 100, fake, 4, 100, 100, 256, 4, fake, None) == 1      # negative count
    assert f(None, 0, 0, None, 0, 0, 100, 256, 4, fake, None) == 0           # nothing to read: no launch


def test_cpu_baseline_states_cores_and_cpu_model():
    sys.path.insert(0, ROOT)
    import bench
    r = bench.cpu_baseline("tiny", 0, 1, budget_s=0.5)
    assert r["kind"] == "oracle" and r["unit"] == "rows/s" and r["value"] > 0
    assert 1 <= r["cores"] <= min(16, r["host_cpus"])
    assert r["host_cpus"] >= 1 and isinstance(r["cpu_model"], str) and r["cpu_model"]
    assert "16" in r["core_cap"]
