"""Plain CPU oracle for confidence-modulated speculative decoding (arXiv 2508.15371).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or link
this module: only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` use it.  It shares no code with the HIP library.

Everything is computed in float64 from the exact input values (bf16 bits or fp32
widened without rounding), with the plainest definition of each quantity: two
passes over a row, ``numpy`` library primitives (max, exp, log, sort, cumsum)
as steps, and no blocking, fusion or reordering.

Each function names the passage it follows.  Readings of passages that the paper
leaves ambiguous are marked "reading"; they are listed with their justification
in the design notes of the repository.

Decisions that turn a floating-point quantity into a discrete outcome (a floor,
an accept/reject comparison, an inverse-CDF index) also return a *slack*: the
distance of the exact quantity from the decision boundary, in the units stated
at each function.  A GPU result that differs from the oracle on a decision whose
slack is below 1e-6 is an allowed, counted exception; any other difference is a
failure.

Parity status: every function here is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_*.py`` and ``tests/test_golden.py``.  Three behaviours marked
"reading" below are choices the paper does not determine; each is pinned to its
reading: the OR of the confidence gate with the stochastic test in CM mode (CM
contains STANDARD, CM with beta = 0 equals it, and the AND of the two fails the
tests), the final sample's own uniform (exact standard speculative sampling over
the whole uniform lattice fails if the rejecting uniform is reused, which biases
the sample), and the zero-residual fallback (a hand-worked case whose residual is
identically zero).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

MODE_STANDARD = 0
MODE_CM = 1
MODE_GREEDY = 2

__all__ = [
    "MODE_STANDARD", "MODE_CM", "MODE_GREEDY", "RowStats", "decode_logits", "row_stats", "logit_variance",
    "normalised_signals", "confidence", "draft_len", "log_softmax_at",
    "stochastic_accept", "top_beta_inclusion", "gap_gate", "accept_position",
    "prefix_length", "residual_pmf", "inverse_cdf", "final_sample", "greedy_next", "draft_sample", "verify_sequence",
]


# ----------------------------------------------------------------------------- inputs
def decode_logits(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored logits: ``dtype`` is "f32" (float32 array) or
    "bf16" (uint16 array of raw bfloat16 bits; value = bits placed in the high half of
    a float32)."""
    if dtype == "f32":
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        b = np.asarray(stored, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return b.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------- Sec. III.B(1)
@dataclass
class RowStats:
    m: float            # max logit z^(1)
    A: float            # sum_v exp(z_v - m)  (softmax normaliser relative to the max)
    H: float            # Shannon entropy of the row's softmax, nats
    top1: int           # lowest index attaining m
    z2: float           # largest logit over all indices except top1 (may equal m, or be -inf)
    p1_minus_p2: float  # softmax margin P^(1) - P^(2)
    margin_logit: float  # z^(1) - z^(2) (+inf when only one finite logit)


def row_stats(z: np.ndarray) -> RowStats:
    """Per-row quantities of the drafter distribution, Sec. III.B(1).

    * Entropy-based confidence: H = -sum_y P(y) log P(y) over the vocabulary,
      with 0 log 0 = 0 (entries at -inf have P = 0).
    * Logit margin: z^(1) - z^(2), top-1 and top-2 logits.
    * Softmax margin: P^(1) - P^(2).

    Reading (ties): the top-1 token is the lowest index attaining the maximum,
    and the top-2 logit is the largest element at any other index, so a repeated
    maximum gives a zero margin.

    Precondition: at least one finite entry; entries may be -inf; no NaN/+inf.
    """
    z = np.asarray(z, dtype=np.float64)
    m = float(z.max())
    e = np.exp(z - m)                 # exp(-inf) = 0
    A = float(e.sum())
    p = e / A
    pos = p > 0
    H = float(-(p[pos] * np.log(p[pos])).sum())
    top1 = int(np.argmax(z))          # first occurrence = lowest index
    z2 = float(np.max(np.delete(z, top1))) if z.size > 1 else -math.inf
    p2 = math.exp(z2 - m) / A if z2 > -math.inf else 0.0
    p1_minus_p2 = float(p[top1]) - p2
    margin_logit = m - z2 if z2 > -math.inf else math.inf
    return RowStats(m, A, H, top1, z2, p1_minus_p2, margin_logit)


def logit_variance(z: np.ndarray) -> float:
    """Population variance of the finite logits of a row: the logit-variance proxy
    for drafter uncertainty that Sec. I names beside entropy and the top-1/top-2
    margin.  The paper gives it no normalisation, so it is reported, not combined
    into C.  Two-pass definition in fp64: the mean first, then the mean squared
    deviation; -inf entries are left out, one finite entry gives 0."""
    z = np.asarray(z, dtype=np.float64)
    f = z[np.isfinite(z)]
    mu = float(f.sum()) / f.size
    return float(((f - mu) ** 2).sum()) / f.size


def normalised_signals(rs: RowStats, V: int, beta_m: float) -> tuple[float, float, float]:
    """The three confidence signals rescaled to [0, 1], Sec. III.B(1).

    * Entropy: the paper rescales H by log|V| (the maximum entropy).  Reading: a
      *confidence* must grow as entropy falls (the draft-length passage says low
      entropy drives the mean confidence towards 1), so the entropy signal is
      1 - H / log|V|.
    * Logit margin: sigmoid(beta_m * (z^(1) - z^(2))), beta_m > 0 a sharpness
      factor (its own symbol here; the paper reuses beta for top-beta).  Since the
      margin is >= 0 this lies in [1/2, 1).  An infinite margin gives 1.
    * Softmax margin: (P^(1) - P^(2)) / (1 - 1/|V|).  Reading: clipped at 1, since
      a one-hot row would otherwise give |V|/(|V|-1) > 1 against the stated [0, 1].
    """
    c_ent = 1.0 - rs.H / math.log(V)
    t = beta_m * rs.margin_logit
    c_margin = 1.0 if t == math.inf else 1.0 / (1.0 + math.exp(-t))
    c_soft = min(1.0, rs.p1_minus_p2 / (1.0 - 1.0 / V))
    return c_ent, c_margin, c_soft


def confidence(rs: RowStats, V: int, lambdas: tuple[float, float, float], beta_m: float) -> float:
    """Unified confidence C = l1*C_ent + l2*C_margin + l3*C_soft, Sec. III.B(1)
    (weights in [0, 1] summing to 1)."""
    c_ent, c_margin, c_soft = normalised_signals(rs, V, beta_m)
    l1, l2, l3 = lambdas
    return l1 * c_ent + l2 * c_margin + l3 * c_soft


# ----------------------------------------------------------------------------- Sec. III.B(b)
def draft_len(C: np.ndarray, k_min: int, k_max: int, alpha: float):
    """Adaptive draft length per sequence, Sec. III.B(b).

    ``C`` is ``[B, k_max]``: the confidence of every drafter position of each
    sequence, available from the speculative pass before the draft length is
    chosen.  Reading (window): the mean runs over all k_max positions.  Reading
    (garbled clip): k = min(k_max, max(k_min, floor(alpha * Cbar * k_max))).

    Returns ``(k[B] int32, offsets[B+1] int32, slack[B])``: offsets is the
    exclusive prefix sum of k_b + 1 (the packed target-row layout: k_b drafted
    positions plus one final position per sequence).  slack_b is the distance of
    alpha*Cbar*k_max from the nearest integer n when the floor there can change
    the clipped result (n in [k_min+1, k_max]), else +inf.

    The mean and product are evaluated left to right in float64:
    s = C_0 + C_1 + ... (sequential), x = alpha * (s / k_max) * k_max.
    """
    C = np.asarray(C, dtype=np.float64)
    B = C.shape[0]
    k = np.empty(B, dtype=np.int32)
    slack = np.empty(B, dtype=np.float64)
    for b in range(B):
        s = 0.0
        for i in range(k_max):
            s += float(C[b, i])
        x = alpha * (s / k_max) * k_max
        k[b] = min(k_max, max(k_min, math.floor(x)))
        n = math.floor(x + 0.5)
        slack[b] = abs(x - n) if k_min + 1 <= n <= k_max else math.inf
    off = np.zeros(B + 1, dtype=np.int64)
    off[1:] = np.cumsum(k.astype(np.int64) + 1)
    return k, off.astype(np.int32), slack


# ----------------------------------------------------------------------------- Sec. III.A / III.B(c)
def log_softmax_at(z: np.ndarray, y: int, rs: RowStats) -> float:
    """log P(y) = (z_y - max) - log(sum exp(z - max)); -inf when z_y = -inf."""
    zy = float(z[y])
    if zy == -math.inf:
        return -math.inf
    return (zy - rs.m) - math.log(rs.A)


def stochastic_accept(u: float, lp_t: float, lp_d: float) -> tuple[bool, float]:
    """Standard speculative-sampling test (the rule of the speculative sampling
    methods the paper cites in Sec. II): accept the drafted token x ~ p_d with
    probability min(1, p_t(x) / p_d(x)), i.e. accept iff u < p_t(x)/p_d(x) for
    u ~ U[0, 1).  Evaluated as log u < log p_t - log p_d.

    Slack: |log u - (log p_t - log p_d)| (log units), +inf if any term is infinite.
    """
    if lp_t == -math.inf:
        return False, math.inf
    if u == 0.0 or lp_d == -math.inf:
        return True, math.inf
    r = lp_t - lp_d
    lu = math.log(u)
    return lu < r, abs(lu - r)


def top_beta_inclusion(z_t: np.ndarray, y: int, beta: int) -> bool:
    """Top-beta inclusion, Sec. III.B(c)(i): log P(y) >= log P(y^(beta)), with
    y^(beta) the beta-th ranked token of the target distribution.

    Log-softmax is the logits shifted by one constant, so the ranking is that of
    the logits: compare z_y with the beta-th largest logit (ties count once per
    element).  beta = 0 never passes; beta > |V| always passes.
    """
    if beta <= 0:
        return False
    if beta > z_t.size:
        return True
    kth = float(np.sort(z_t)[::-1][beta - 1])
    return float(z_t[y]) >= kth


def gap_gate(z_t: np.ndarray, y: int, rs_t: RowStats, tau: float) -> tuple[bool, float, float]:
    """Gap-bounded acceptance, Sec. III.B(c)(ii): log P(y^(1)) - log P(y) <= tau_t.

    The normaliser cancels, so the gap is z^(1) - z_y exactly.  Returns
    (passes, gap, slack = |gap - tau|)."""
    zy = float(z_t[y])
    gap = rs_t.m - zy if zy > -math.inf else math.inf
    ok = gap <= tau
    return ok, gap, (abs(gap - tau) if math.isfinite(gap) else math.inf)


def accept_position(z_t: np.ndarray, rs_t: RowStats, z_d: np.ndarray, rs_d: RowStats, y: int,
                    u: float, C: float, mode: int, beta: int, tau_base: float, gamma: float) -> dict:
    """Acceptance of one drafted position.

    * Adaptive threshold tau_t = tau_base + gamma * (1 - C_t), Sec. III.B(c).
    * Gate = top-beta inclusion AND gap <= tau_t, Sec. III.B(c) "modified
      verification rule".
    * Reading (the paper does not fix it): the paper's gate relaxes acceptance, so in CM mode
      a position is accepted when the stochastic test passes OR the gate passes;
      in STANDARD mode only the stochastic test applies (standard speculative
      sampling).
    * GREEDY mode is the paper's deterministic verification (Sec. III.A step 2)
      with the gate as its relaxation: accepted iff the draft is the target's top
      token (lowest index among equal maxima) OR the gate passes; no uniform is
      consumed.  With beta = 0 (gate off) this is exact-match verification.

    Returns a dict with acc, stoch, gate, n_greater_clamped (= min(#{v: z_v > z_y},
    beta)), and the slacks of the two inexact sub-decisions.
    """
    lp_t = log_softmax_at(z_t, y, rs_t)
    lp_d = log_softmax_at(z_d, y, rs_d)
    stoch, s_stoch = stochastic_accept(u, lp_t, lp_d)
    tau = tau_base + gamma * (1.0 - C)
    rank_ok = top_beta_inclusion(z_t, y, beta)
    gap_ok, gap, s_gap = gap_gate(z_t, y, rs_t, tau)
    gate = rank_ok and gap_ok
    exact = y == int(np.argmax(z_t))
    if mode == MODE_GREEDY:
        acc = exact or gate
    else:
        acc = stoch or (mode == MODE_CM and gate)
    n_greater = int(np.count_nonzero(z_t > z_t[y]))
    return {
        "acc": acc, "stoch": stoch, "gate": gate, "exact": exact, "rank_ok": rank_ok, "gap_ok": gap_ok,
        "gap": gap, "tau": tau, "lp_t": lp_t, "lp_d": lp_d,
        "slack_stoch": s_stoch if mode != MODE_GREEDY else math.inf,
        "slack_gap": s_gap if mode in (MODE_CM, MODE_GREEDY) and rank_ok else math.inf,
        "n_greater_clamped": min(n_greater, max(beta, 0)),
    }


def prefix_length(flags) -> int:
    """Accepted prefix c: verification halts at the first rejected position and
    discards the rest (Sec. III.A step 2; Sec. III.B(c) modified rule)."""
    for i, f in enumerate(flags):
        if not f:
            return i
    return len(flags)


def residual_pmf(z_t: np.ndarray, rs_t: RowStats, z_d: np.ndarray, rs_d: RowStats) -> np.ndarray:
    """Unnormalised residual max(0, p_t - p_d) after a rejection (standard
    speculative sampling).  Reading (the paper does not fix it): if it is
    identically zero (through rounding, or when drafter and target rows are equal
    and the draft was a token both rows mask), p_t is used instead."""
    p_t = np.exp(z_t - rs_t.m) / rs_t.A
    p_d = np.exp(z_d - rs_d.m) / rs_d.A
    q = np.maximum(0.0, p_t - p_d)
    if not np.any(q > 0):
        return p_t
    return q


def inverse_cdf(q: np.ndarray, u: float) -> tuple[int, float]:
    """Sample index y from the unnormalised pmf q with the uniform u in [0, 1):
    the smallest y whose cumulative sum (sequential, vocabulary order) exceeds
    u * R, R the total; if rounding leaves none, the last y with q_y > 0.

    Slack: min(u*R - CDF(y-1), CDF(y) - u*R) / R."""
    c = np.cumsum(np.asarray(q, dtype=np.float64))
    R = float(c[-1])
    x = u * R
    hit = np.nonzero(c > x)[0]
    if hit.size:
        y = int(hit[0])
    else:
        y = int(np.nonzero(q > 0)[0][-1])
    lo = float(c[y - 1]) if y > 0 else 0.0
    hi = float(c[y])
    return y, min(x - lo, hi - x) / R


def final_sample(z_t_rows: list, rs_t_rows: list, z_d_rows: list, rs_d_rows: list,
                 k_b: int, n_acc: int, u_final: float) -> tuple[int, float]:
    """The token emitted after the accepted prefix: on a rejection at position
    c = n_acc < k_b, a sample from the residual of target and drafter rows c;
    when all k_b drafts are accepted, a sample from the target row k_b (the row
    scored after the last draft).  Reading (the paper does not fix it): this sample
    uses the sequence's own final uniform (slot k_b), not the rejecting one."""
    if n_acc < k_b:
        q = residual_pmf(z_t_rows[n_acc], rs_t_rows[n_acc], z_d_rows[n_acc], rs_d_rows[n_acc])
    else:
        t = z_t_rows[k_b]
        q = np.exp(t - rs_t_rows[k_b].m) / rs_t_rows[k_b].A
    return inverse_cdf(q, u_final)


def greedy_next(z_t_rows: list, k_b: int, n_acc: int) -> int:
    """GREEDY mode's final token: the target's top token (lowest index among equal
    maxima) at the first rejected position, or at position k_b when every draft
    passed -- the verifier's own autoregressive choice ("reprocessed via AR
    decoding", Sec. III.B(c); Sec. III.A step 2)."""
    return int(np.argmax(z_t_rows[min(n_acc, k_b)]))


def draft_sample(z: np.ndarray, u: float) -> tuple[int, float]:
    """A sampled draft: x ~ p_d = softmax(z), by the inverse CDF with u (the
    convention of ``inverse_cdf``).  Speculative sampling's exactness assumes drafts
    drawn this way; the paper's drafter itself takes the argmax (Sec. III.A step 1)."""
    rs = row_stats(z)
    return inverse_cdf(np.exp(np.asarray(z, dtype=np.float64) - rs.m) / rs.A, u)


def verify_sequence(z_t_rows: list, z_d_rows: list, drafted, uniforms, C, k_b: int, mode: int,
                    beta: int, tau_base: float, gamma: float, n_acc_override: int | None = None) -> dict:
    """Verify one sequence: positions 0..k_b-1 against target rows 0..k_b-1, then
    the final sample.  ``z_t_rows`` has k_b+1 rows, ``z_d_rows`` at least k_b
    rows (and row n_acc when n_acc < k_b), ``uniforms`` k_b+1 values (slot k_b
    for the final sample), ``C`` the drafter confidences.

    ``n_acc_override`` lets a parity test take the final sample after a given
    prefix length (stage isolation when an upstream low-slack decision differs).
    """
    rs_t = [row_stats(t) for t in z_t_rows[:k_b + 1]]
    rs_d = [row_stats(d) for d in z_d_rows[:k_b]]
    pos = []
    for i in range(k_b):
        pos.append(accept_position(z_t_rows[i], rs_t[i], z_d_rows[i], rs_d[i], int(drafted[i]),
                                   float(uniforms[i]), float(C[i]), mode, beta, tau_base, gamma))
    flags = [p["acc"] for p in pos]
    n_acc = prefix_length(flags)
    c = n_acc if n_acc_override is None else n_acc_override
    if mode == MODE_GREEDY:
        nxt, s_nxt = greedy_next(z_t_rows, k_b, c), math.inf
    else:
        nxt, s_nxt = final_sample(z_t_rows, rs_t, z_d_rows, rs_d, k_b, c, float(uniforms[k_b]))
    return {"positions": pos, "flags": flags, "n_acc": n_acc, "next": nxt, "slack_next": s_nxt,
            "rs_t": rs_t, "rs_d": rs_d}
