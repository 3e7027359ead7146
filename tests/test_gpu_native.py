"""A native consumer of the C ABI (tests/native/logit_pass_native.cpp: C++ on the HIP
runtime, no Python or torch) runs one decoding iteration by the three calls and by
cmsd_logit_pass on device buffers it allocates itself, requires the two to agree bit
for bit, and writes its seeded inputs and outputs; here they are checked against
the oracle (drafter stats, draft lengths, accept tests, prefixes, final tokens)."""
import os
import subprocess

import numpy as np
import pytest

from oracle import cmsd_oracle as O
from tests import harness as Hn

pytestmark = pytest.mark.gpu
BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "logit_pass_native")


def _read(path):
    raw = open(path, "rb").read()
    B, K, V = np.frombuffer(raw[:12], dtype=np.int32)
    B, K, V = int(B), int(K), int(V)
    out, pos = {}, 12
    for name, dt, n in (("zd", np.float32, B * K * V), ("zt", np.float32, B * (K + 1) * V),
                        ("drafted", np.int32, B * K), ("unif", np.float32, B * (K + 1)),
                        ("stats", np.float32, B * K * 8), ("tstats", np.float32, B * (K + 1) * 8),
                        ("k", np.int32, B), ("n_acc", np.int32, B), ("next", np.int32, B)):
        a = np.frombuffer(raw, dtype=dt, count=n, offset=pos)
        pos += a.nbytes
        out[name] = a
    assert pos == len(raw)
    return B, K, V, out


def test_native_consumer_matches_oracle(tmp_path):
    if not os.path.exists(BIN):
        pytest.fail(f"{BIN} is not built (python -m paper_2508_15371_amd.build builds it with the library)")
    path = os.path.join(str(tmp_path), "native.bin")
    r = subprocess.run([BIN, path], capture_output=True, text=True, timeout=120)
    print(r.stdout.strip(), flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    B, K, V, d = _read(path)
    import torch
    gs = Hn.stats_np(torch.from_numpy(d["stats"].reshape(B * K, 8).copy()))
    ts = Hn.tstats_np(torch.from_numpy(d["tstats"].reshape(B * (K + 1), 8).copy()))
    zd = d["zd"].reshape(B * K, V)
    zt = d["zt"].reshape(B * (K + 1), V)
    drafted = d["drafted"].reshape(B, K)
    unif = d["unif"].reshape(B, K + 1)
    P = Hn.PARAMS
    lam = tuple(Hn.f32(x) for x in P["lambdas"])
    t = Hn.Tally()
    # draft lengths from the GPU's confidences: bit-exact
    k_o, _, _ = O.draft_len(gs["C"].astype(np.float64).reshape(B, K), P["k_min"], K, Hn.f32(P["alpha"]))
    t.value("k(stage)", np.array_equal(k_o, d["k"]), (k_o, d["k"]))
    for b in range(B):
        zdb = [Hn.decode(zd[b * K + i], "f32") for i in range(K)]
        for i in range(K):
            Hn.check_row_stats(t, gs, b * K + i, zdb[i], V, lam, Hn.f32(P["beta_margin"]))
        C = [O.confidence(O.row_stats(z), V, lam, Hn.f32(P["beta_margin"])) for z in zdb]
        ztb = [Hn.decode(zt[b * (K + 1) + i], "f32") for i in range(K + 1)]
        Hn.check_sequence(t, b, ztb, zdb, drafted[b], [float(u) for u in unif[b]], C, K, O.MODE_CM, P, ts,
                          b * (K + 1), int(d["n_acc"][b]), int(d["next"][b]))
    print(f"[native parity] checked={t.checked} exceptions={t.exceptions}", flush=True)
    t.assert_ok()
