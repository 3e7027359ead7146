"""The oracle's pins catch plausible mistakes (CPU only): each mistake below is
planted in a copy of the oracle in a scratch directory, and the pin tests
(tests/test_oracle_*.py and the hand-worked example) must then fail.  The
repository's own oracle is never modified."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["test_oracle_stats.py", "test_oracle_draft_len.py", "test_oracle_verify.py", "test_golden.py"]
HELPERS = ["__init__.py", "conftest.py", "golden_example.py"]

# (text in oracle/cmsd_oracle.py, the mistake, what it breaks)
MUTATIONS = [
    ("H = float(-(p[pos] * np.log(p[pos])).sum())", "H = float(-(p[pos] * np.log(p[pos])).sum()) + 1e-9",
     "entropy offset"),
    ("c_ent = 1.0 - rs.H / math.log(V)", "c_ent = rs.H / math.log(V)", "entropy signal direction"),
    ("1.0 / (1.0 + math.exp(-t))", "1.0 / (1.0 + math.exp(t))", "logit-margin sigmoid sign"),
    ("rs.p1_minus_p2 / (1.0 - 1.0 / V)", "rs.p1_minus_p2 / (1.0 - 1.0 / (V - 1))", "softmax-margin normaliser"),
    ("k[b] = min(k_max, max(k_min, math.floor(x)))", "k[b] = min(k_max, max(k_min, math.ceil(x)))",
     "floor vs ceil in the draft length"),
    ("        x = alpha * (s / k_max) * k_max\n", "        x = alpha * (s / (k_max + 1)) * k_max\n",
     "mean over the wrong window"),
    ("return lu < r, abs(lu - r)", "return lu < -r, abs(lu - r)", "accept-ratio direction"),
    ("return float(z_t[y]) >= kth", "return float(z_t[y]) > kth", ">= vs > in top-beta"),
    ("tau = tau_base + gamma * (1.0 - C)", "tau = tau_base + gamma * C", "threshold uses C, not 1 - C"),
    ("acc = stoch or (mode == MODE_CM and gate)", "acc = stoch and (mode == MODE_CM and gate) or stoch and mode != MODE_CM",
     "gate AND-ed instead of OR-ed"),
    ("q = np.maximum(0.0, p_t - p_d)", "q = np.maximum(0.0, p_d - p_t)", "residual sign"),
    ("t = z_t_rows[k_b]", "t = z_t_rows[k_b - 1]", "bonus row index"),
    ("hit = np.nonzero(c > x)[0]", "hit = np.nonzero(c >= x)[0]", ">= vs > in the inverse CDF"),
    ("top1 = int(np.argmax(z))  ", "top1 = int(z.size - 1 - np.argmax(z[::-1]))  ", "highest instead of lowest max index"),
    ("p1_minus_p2 = float(p[top1]) - p2", "p1_minus_p2 = float(p[top1]) + p2", "softmax-margin sign"),
    ("off[1:] = np.cumsum(k.astype(np.int64) + 1)", "off[1:] = np.cumsum(k.astype(np.int64))",
     "offsets without the final row"),
    ("gap = rs_t.m - zy if", "gap = zy - rs_t.m if", "gap sign"),
    ("exact = y == int(np.argmax(z_t))", "exact = y == int(np.argmax(z_t)) or y == 0", "GREEDY exact-match test"),
    ("            return i\n", "            return i + 1\n", "prefix keeps the first rejected draft"),
    ("p_d = np.exp(z_d - rs_d.m) / rs_d.A", "p_d = np.exp(z_d - rs_d.m) / rs_t.A",
     "residual with the target's normaliser on the drafter row"),
    ("return int(np.argmax(z_t_rows[min(n_acc, k_b)]))", "return int(np.argmax(z_t_rows[k_b]))",
     "GREEDY final token from the bonus row after a rejection"),
    ("k_b, c, float(uniforms[k_b]))", "k_b, c, float(uniforms[min(c, k_b)]))",
     "final sample reuses the rejecting position's uniform"),
    ("    if not np.any(q > 0):\n        return p_t\n", "", "no fallback for a zero residual"),
    ("    if not np.any(q > 0):\n        return p_t\n", "    if not np.any(q > 0):\n        return np.ones_like(p_t)\n",
     "uniform fallback for a zero residual"),
]


def _scratch_copy(dst):
    ign = shutil.ignore_patterns("__pycache__", "*.pyc")
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(dst, "oracle"), ignore=ign)
    shutil.copytree(os.path.join(ROOT, "workloads"), os.path.join(dst, "workloads"), ignore=ign)
    os.makedirs(os.path.join(dst, "tests"))
    for f in HELPERS + PINS:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(dst, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(dst, "tests", "golden"))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), dst)


def _run_pins(cwd):
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           *[os.path.join("tests", f) for f in PINS]],
                          cwd=cwd, capture_output=True, text=True, timeout=900)


def _mutated_run(base, idx):
    """Run the pins against a scratch copy of the oracle carrying mutation idx
    (idx = -1: the unmodified oracle); returns (returncode, output tail)."""
    d = os.path.join(base, f"m{idx}")
    _scratch_copy(d)
    if idx >= 0:
        orig, mutant, what = MUTATIONS[idx]
        path = os.path.join(d, "oracle", "cmsd_oracle.py")
        src = open(path).read()
        if src.count(orig) != 1:
            return -1, f"the oracle no longer contains the line for: {what}"
        with open(path, "w") as f:
            f.write(src.replace(orig, mutant))
    r = _run_pins(d)
    return r.returncode, r.stdout[-3000:]


@pytest.fixture(scope="module")
def runs(tmp_path_factory):
    """Every mutated copy (and the unmodified one) runs the pins, in parallel."""
    from concurrent.futures import ThreadPoolExecutor
    base = str(tmp_path_factory.mktemp("oracle_mutations"))
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count() or 1
    idx = list(range(-1, len(MUTATIONS)))
    with ThreadPoolExecutor(max(1, min(8, ncpu))) as ex:
        return dict(zip(idx, ex.map(lambda i: _mutated_run(base, i), idx)))


def test_unmodified_copy_passes(runs):
    rc, out = runs[-1]
    assert rc == 0, out


@pytest.mark.parametrize("i", range(len(MUTATIONS)), ids=[m[2] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(runs, i):
    rc, out = runs[i]
    assert rc == 1, f"no pin caught: {MUTATIONS[i][2]}\n{out}"
