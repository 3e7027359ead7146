"""The comparison rules of the parity tests, for numpy arrays of the GPU's outputs:
values within their tolerance, decisions equal unless the oracle's slack for that
decision is below SLACK (an allowed, counted exception).  Imports numpy and the oracle
only (no torch), so worker processes that check a batch in parallel load it cheaply."""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from oracle import cmsd_oracle as O

SLACK = 1e-6          # decision slack below which a GPU/oracle difference is an exception
REL = 1e-4            # entropy / margin / confidence tolerance: |d| <= REL * max(|ref|, 1e-2)
PARAMS = dict(lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin=1.0, k_min=1, alpha=1.0, top_beta=3,
              tau_base=0.1, gamma=1.0)


def f32(x) -> float:
    """Value of x rounded to float32 (the parameter the device sees), as a Python float."""
    return float(np.float32(x))


def decode(stored: np.ndarray, dtype: str) -> np.ndarray:
    return O.decode_logits(stored, dtype)


def close_rel(gpu: float, ref: float, rel: float = REL, floor: float = 1e-2) -> bool:
    if math.isinf(ref) or math.isinf(gpu):
        return gpu == ref
    return abs(gpu - ref) <= rel * max(abs(ref), floor)


@dataclass
class Tally:
    checked: int = 0
    exceptions: int = 0
    failures: list = field(default_factory=list)

    def decision(self, name: str, gpu, ref, slack: float) -> None:
        self.checked += 1
        if gpu == ref:
            return
        if slack < SLACK:
            self.exceptions += 1
        else:
            self.failures.append((name, gpu, ref, slack))

    def value(self, name: str, ok: bool, detail) -> None:
        self.checked += 1
        if not ok:
            self.failures.append((name, detail))

    def assert_ok(self) -> None:
        assert not self.failures, f"{len(self.failures)} failures (of {self.checked}); first: {self.failures[:5]}"


def check_row_stats(t: Tally, g: dict, r: int, z: np.ndarray, V: int, lam, beta_m) -> O.RowStats:
    """Compare GPU drafter stats row r with the oracle on logits z."""
    rs = O.row_stats(z)
    C = O.confidence(rs, V, lam, beta_m)
    t.value(f"m[{r}]", g["m"][r] == np.float32(rs.m), (g["m"][r], rs.m))
    t.value(f"top1[{r}]", int(g["top1"][r]) == rs.top1, (int(g["top1"][r]), rs.top1))
    t.value(f"mlogit[{r}]", close_rel(float(g["mlogit"][r]), rs.margin_logit, 1e-6, 1e-30),
            (float(g["mlogit"][r]), rs.margin_logit))
    t.value(f"A[{r}]", close_rel(float(g["A"][r]), rs.A, 1e-5, 0.0), (float(g["A"][r]), rs.A))
    t.value(f"H[{r}]", close_rel(float(g["H"][r]), rs.H), (float(g["H"][r]), rs.H))
    t.value(f"msoft[{r}]", close_rel(float(g["msoft"][r]), rs.p1_minus_p2), (float(g["msoft"][r]), rs.p1_minus_p2))
    t.value(f"C[{r}]", close_rel(float(g["C"][r]), C), (float(g["C"][r]), C))
    has_ninf = bool(np.any(z == -math.inf))
    t.value(f"flags[{r}]", (int(g["flags"][r]) & 1) == int(has_ninf), (int(g["flags"][r]), has_ninf))
    return rs


def acc_allowed(p: dict, mode: int) -> set:
    """acc values reachable by flipping sub-decisions whose slack is below SLACK."""
    stochs = {p["stoch"]} | ({not p["stoch"]} if p["slack_stoch"] < SLACK else set())
    gaps = {p["gap_ok"]} | ({not p["gap_ok"]} if p["slack_gap"] < SLACK else set())
    if mode == O.MODE_GREEDY:
        return {p["exact"] or (p["rank_ok"] and gg) for gg in gaps}
    return {s or (mode == O.MODE_CM and p["rank_ok"] and gg) for s in stochs for gg in gaps}


def check_sequence(t: Tally, b: int, zt_rows, zd_rows, drafted, unif, C, kb: int, mode: int, prm: dict,
                   ts: dict, toff: int, n_acc_gpu: int, next_gpu: int) -> None:
    """Compare one sequence's verify outputs; the oracle takes the final sample after
    the GPU's prefix length (stage isolation of an upstream low-slack flip)."""
    res = O.verify_sequence(zt_rows, zd_rows, drafted, unif, C, kb, mode, prm["top_beta"],
                            f32(prm["tau_base"]), f32(prm["gamma"]), n_acc_override=n_acc_gpu)
    flags_gpu = []
    for i in range(kb + 1):
        rs = res["rs_t"][i]
        t.value(f"tm[{b},{i}]", ts["m"][toff + i] == np.float32(rs.m), (ts["m"][toff + i], rs.m))
        t.value(f"tA[{b},{i}]", close_rel(float(ts["A"][toff + i]), rs.A, 1e-5, 0.0), (ts["A"][toff + i], rs.A))
    t.value(f"final-row[{b}]", int(ts["acc"][toff + kb]) == -1, int(ts["acc"][toff + kb]))
    if mode == O.MODE_GREEDY:
        for i in range(kb + 1):
            want = int(np.argmax(zt_rows[i]))
            t.value(f"top1[{b},{i}]", int(ts["top1"][toff + i]) == want, (int(ts["top1"][toff + i]), want))
    for i in range(kb):
        p = res["positions"][i]
        a = int(ts["acc"][toff + i])
        flags_gpu.append(a == 1)
        t.checked += 1
        if a not in (0, 1):
            t.failures.append((f"acc[{b},{i}] invalid", a))
        elif (a == 1) != p["acc"]:
            if (a == 1) in acc_allowed(p, mode):
                t.exceptions += 1
            else:
                t.failures.append((f"acc[{b},{i}]", a, p))
        if mode in (O.MODE_CM, O.MODE_GREEDY) and prm["top_beta"] > 0:
            t.value(f"ngt[{b},{i}]", int(ts["ngt"][toff + i]) == p["n_greater_clamped"],
                    (int(ts["ngt"][toff + i]), p["n_greater_clamped"]))
    want = O.prefix_length(flags_gpu)
    t.value(f"n_acc-vs-own-flags[{b}]", n_acc_gpu == want, (n_acc_gpu, want))
    if n_acc_gpu != res["n_acc"]:
        # must follow from excepted flag flips
        t.checked += 1
        t.exceptions += 1
    t.decision(f"next[{b}]", next_gpu, res["next"], res["slack_next"])


def oracle_conf(z: np.ndarray, V: int) -> float:
    lam = tuple(f32(x) for x in PARAMS["lambdas"])
    return O.confidence(O.row_stats(z), V, lam, f32(PARAMS["beta_margin"]))


def stats_fields(f: np.ndarray, i: np.ndarray) -> dict:
    """Named columns of drafter stats records given as float32 [n, 8] and its int32 view."""
    return {"m": f[:, 0], "A": f[:, 1], "H": f[:, 2], "msoft": f[:, 3], "mlogit": f[:, 4], "C": f[:, 5],
            "top1": i[:, 6], "flags": i[:, 7]}


def tstats_fields(f: np.ndarray, i: np.ndarray) -> dict:
    """Named columns of target-row records given as float32 [n, 8] and its int32 view."""
    return {"m": f[:, 0], "A": f[:, 1], "ngt": i[:, 2], "acc": i[:, 3], "top1": i[:, 4]}
