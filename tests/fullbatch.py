"""Whole-batch parity: every sequence of a workload checked against the oracle, the
oracle's work spread over forked worker processes (numpy only; they inherit the
host arrays of the workload and the GPU's outputs from the parent, copy-on-write).

The parent sets the job with ``set_job`` and then creates the pool, so every worker
sees that job; ``check_batch`` splits the sequences over the pool and sums the tallies.
"""
from __future__ import annotations

import multiprocessing as mp
import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from oracle import cmsd_oracle as O
from tests import parity as Pa

_JOB: dict = {}


def workers() -> int:
    """Worker processes: the host's cores, at most 16 (one GPU's share of its host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def set_job(**job) -> None:
    """cfg, draft/target/drafted/uniforms (host arrays of the workload, dense by
    sequence), gs (drafter stats fields, all rows), ts (target-row record fields, rows
    as the GPU wrote them), k, n_acc, next (per sequence), off (first target row of
    each sequence in ``ts``), packed (bool: target rows were packed by k),
    verify_len ("k_max", "k_b"), mode, params."""
    _JOB.clear()
    _JOB.update(job)


def _check_seqs(seqs) -> tuple[int, int, list, float]:
    j = _JOB
    cfg, P, mode = j["cfg"], j["params"], j["mode"]
    K, V, dt = cfg.k_max, cfg.V, cfg.dtype
    lam = tuple(Pa.f32(x) for x in P["lambdas"])
    bm = Pa.f32(P["beta_margin"])
    t = Pa.Tally()
    for b in seqs:
        zd = [Pa.decode(j["draft"][b * K + i], dt) for i in range(K)]
        # every drafter row's record (Sec. III.B(1))
        C = []
        for i in range(K):
            rs = Pa.check_row_stats(t, j["gs"], b * K + i, zd[i], V, lam, bm)
            C.append(O.confidence(rs, V, lam, bm))
        # the draft length from the oracle's own confidences (Sec. III.B(b))
        kb_o, _, sl = O.draft_len(np.array([C]), P["k_min"], K, Pa.f32(P["alpha"]))
        t.decision(f"k[{b}]", int(j["k"][b]), int(kb_o[0]), float(sl[0]))
        # verification of the positions the GPU verified (its own draft length: stage
        # isolation of an excepted floor flip), Sec. III.A / III.B(c)
        kv = int(j["k"][b]) if j["verify_len"] == "k_b" else K
        toff = int(j["off"][b])
        pos = list(range(kv)) + [K if j["packed"] else kv]
        zt = [Pa.decode(j["target"][b * (K + 1) + i], dt) for i in pos]
        unif = [float(j["uniforms"][b, i]) for i in pos]
        Pa.check_sequence(t, b, zt, zd, j["drafted"][b], unif, C, kv, mode, P, j["ts"], toff, int(j["n_acc"][b]),
                          int(j["next"][b]))
    return t.checked, t.exceptions, t.failures[:20], len(t.failures)


def check_batch(seqs=None) -> Pa.Tally:
    """Check the current job's sequences (all of them by default) over a fork pool."""
    B = _JOB["cfg"].B
    seqs = list(range(B)) if seqs is None else list(seqs)
    n = workers()
    chunks = [c.tolist() for c in np.array_split(np.array(seqs, dtype=np.int64), min(len(seqs), 4 * n)) if len(c)]
    total = Pa.Tally()
    nfail = 0
    with ProcessPoolExecutor(n, mp_context=mp.get_context("fork")) as ex:
        for checked, exc, fails, nf in ex.map(_check_seqs, chunks):
            total.checked += checked
            total.exceptions += exc
            total.failures.extend(fails[: max(0, 20 - len(total.failures))])
            nfail += nf
    total.n_failures = nfail
    return total
