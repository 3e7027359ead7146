"""Pins of the oracle's verification step (Sec. III.A, III.B(c)) and of the
standard speculative-sampling rule it reduces to when modulation is off.

The central pin is exact enumeration: with modulation off, drafting from p_d and
verifying must emit tokens distributed exactly as the target rows p_t.  The test
enumerates every drafted sequence (weight prod p_d) and integrates every uniform
exactly over the 2^24-point lattice the workloads draw uniforms from, locating
each decision boundary by bisection on the oracle's own ``verify_sequence``
(its decisions are monotone in each uniform).  CPU only.
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special

from oracle import cmsd_oracle as O

N = 1 << 24


def u_at(j: int) -> float:
    return j * 2.0 ** -24


def first_true(pred) -> int:
    """Smallest j in [0, N] with pred(j) True for a monotone False..True predicate (N if none)."""
    lo, hi = 0, N
    while lo < hi:
        mid = (lo + hi) // 2
        if pred(mid):
            hi = mid
        else:
            lo = mid + 1
    return lo


def softmax(z):
    return scipy.special.softmax(np.asarray(z, dtype=np.float64))


def _rows(g, V, n, mask_prob=0.15):
    rows = []
    for _ in range(n):
        z = g.normal(0, float(g.uniform(0.3, 2.5)), V)
        m = g.random(V) < mask_prob
        m[int(np.argmax(z))] = False
        z[m] = -math.inf
        rows.append(z)
    return rows


# ----------------------------------------------------------------------------- building blocks
@pytest.mark.parametrize("seed", range(8))
def test_inverse_cdf_exact_measure(seed):
    g = np.random.default_rng(seed)
    V = int(g.integers(1, 9))
    q = g.random(V) * (g.random(V) < 0.7)
    if not (q > 0).any():
        q[int(g.integers(0, V))] = 0.3
    pos = np.nonzero(q > 0)[0]
    assert O.inverse_cdf(q, 0.0)[0] == pos[0]
    assert O.inverse_cdf(q, 1.0 - 2.0 ** -24)[0] == pos[-1]
    starts = [first_true(lambda j, y=y: O.inverse_cdf(q, u_at(j))[0] >= y) for y in range(V)] + [N]
    for y in range(V):
        meas = (starts[y + 1] - starts[y]) / N
        assert meas == pytest.approx(q[y] / q.sum(), abs=2.0 / N)
        if q[y] == 0:
            assert meas == 0


@pytest.mark.parametrize("ratio", [0.0, 1e-3, 0.2, 0.5, 0.999, 1.0, 3.0])
def test_stochastic_accept_measure(ratio):
    lp_d = math.log(0.4)
    lp_t = math.log(0.4 * ratio) if ratio > 0 else -math.inf
    j = first_true(lambda j: not O.stochastic_accept(u_at(j), lp_t, lp_d)[0])
    assert j / N == pytest.approx(min(1.0, ratio), abs=1.0 / N)


def test_stochastic_accept_edge_cases():
    assert O.stochastic_accept(0.0, math.log(0.1), math.log(0.9))[0]
    assert not O.stochastic_accept(0.0, -math.inf, math.log(0.9))[0]
    assert O.stochastic_accept(0.99, math.log(0.1), -math.inf)[0]


@pytest.mark.parametrize("seed", range(30))
def test_top_beta_inclusion_brute_force(seed):
    # rank by counting strictly larger logits (ties share a rank)
    g = np.random.default_rng(seed)
    V = int(g.integers(1, 9))
    z = g.integers(-2, 3, V).astype(np.float64)
    for y in range(V):
        greater = sum(1 for v in range(V) if z[v] > z[y])
        for beta in range(0, V + 2):
            assert O.top_beta_inclusion(z, y, beta) == (greater < beta)


@pytest.mark.parametrize("seed", range(5))
def test_gap_is_log_prob_gap(seed):
    g = np.random.default_rng(seed)
    z = g.normal(0, 2, 300)
    rs = O.row_stats(z)
    lp = scipy.special.log_softmax(z)
    for y in g.integers(0, 300, 10):
        ok, gap, _ = O.gap_gate(z, int(y), rs, 1.0)
        assert gap == pytest.approx(lp.max() - lp[y], abs=1e-12)
        assert ok == (gap <= 1.0)
        assert O.log_softmax_at(z, int(y), rs) == pytest.approx(lp[y], abs=1e-12)


def test_prefix_length_brute_force():
    # leading run of accepted positions, by a cumulative product
    for k in range(0, 13):
        for bits in range(1 << k):
            flags = [bool((bits >> i) & 1) for i in range(k)]
            want = int(np.cumprod(np.array(flags, dtype=np.int64)).sum()) if k else 0
            assert O.prefix_length(flags) == want


# ----------------------------------------------------------------------------- exactness theorem
def _exact_emission_distribution(zt, zd, k, mode=O.MODE_STANDARD, beta=3, tau_base=0.1, gamma=1.0, C=None):
    """Exact distribution of the emitted sequence (accepted drafts + final token)."""
    V = zt[0].size
    C = C if C is not None else [0.5] * k
    pd = [softmax(z) for z in zd]
    dist = {}
    for ys in itertools.product(range(V), repeat=k):
        w = 1.0
        for i, y in enumerate(ys):
            w *= pd[i][y]
        if w == 0.0:
            continue

        def run(us, uf):
            return O.verify_sequence(zt, zd, ys, list(us) + [uf], C, k, mode, beta, tau_base, gamma)

        # accept threshold of each position, by bisection on its own uniform
        thr = []
        for i in range(k):
            def rejects(j, i=i):
                us = [0.0] * k
                us[i] = u_at(j)
                return not run(us, 0.0)["flags"][i]
            thr.append(first_true(rejects))
        for c in range(k + 1):
            p = w
            for i in range(c):
                p *= thr[i] / N
            if c < k:
                p *= 1.0 - thr[c] / N
            if p == 0.0:
                continue
            us = [0.0] * k
            if c < k:
                us[c] = u_at(thr[c])
            assert run(us, 0.0)["n_acc"] == c
            starts = [first_true(lambda j, y=y: run(us, u_at(j))["next"] >= y) for y in range(V)] + [N]
            for y in range(V):
                mass = (starts[y + 1] - starts[y]) / N
                if mass:
                    key = tuple(ys[:c]) + (y,)
                    dist[key] = dist.get(key, 0.0) + p * mass
    return dist


@pytest.mark.parametrize("V,k,seed", [(4, 1, 0), (6, 1, 1), (8, 1, 2), (5, 2, 3), (4, 2, 4), (4, 3, 5), (3, 3, 6)])
def test_standard_mode_emits_target_distribution(V, k, seed):
    g = np.random.default_rng(100 + seed)
    zd = _rows(g, V, k)
    zt = _rows(g, V, k + 1)
    pt = [softmax(z) for z in zt]
    dist = _exact_emission_distribution(zt, zd, k)
    assert sum(dist.values()) == pytest.approx(1.0, abs=1e-9)
    # every emitted position j, conditioned on the emitted prefix, follows p_t,j
    for j in range(k + 1):
        prefixes = {}
        for e, pr in dist.items():
            if len(e) > j:
                prefixes.setdefault(e[:j], np.zeros(V))[e[j]] += pr
        for pre, vec in prefixes.items():
            tot = vec.sum()
            if tot < 1e-6:
                continue
            np.testing.assert_allclose(vec / tot, pt[j], atol=4e-6 / tot)


def test_cm_mode_relaxes_acceptance():
    # the gate only adds acceptances; with beta = 0 (gate off) CM equals STANDARD;
    # gamma = 0 makes the threshold independent of the confidence (fixed tau)
    g = np.random.default_rng(9)
    V, k = 50, 6
    for trial in range(20):
        zd = _rows(g, V, k, 0.0)
        zt = _rows(g, V, k + 1, 0.0)
        ys = [int(np.argmax(z + g.gumbel(size=V))) for z in zd]
        us = g.random(k + 1).tolist()
        C = g.random(k).tolist()
        st = O.verify_sequence(zt, zd, ys, us, C, k, O.MODE_STANDARD, 3, 0.1, 1.0)
        cm = O.verify_sequence(zt, zd, ys, us, C, k, O.MODE_CM, 3, 0.1, 1.0)
        off = O.verify_sequence(zt, zd, ys, us, C, k, O.MODE_CM, 0, 0.1, 1.0)
        assert off["flags"] == st["flags"] and off["next"] == st["next"]
        for a, b in zip(st["flags"], cm["flags"]):
            assert b or not a
        assert cm["n_acc"] >= st["n_acc"]
        f1 = O.verify_sequence(zt, zd, ys, us, C, k, O.MODE_CM, 3, 0.4, 0.0)
        f2 = O.verify_sequence(zt, zd, ys, us, [0.0] * k, k, O.MODE_CM, 3, 0.4, 0.0)
        assert f1["flags"] == f2["flags"]
        for p in f1["positions"]:
            assert p["tau"] == 0.4
        # a huge threshold with beta >= |V| accepts everything
        allacc = O.verify_sequence(zt, zd, ys, us, C, k, O.MODE_CM, V, 1e9, 0.0)
        assert allacc["n_acc"] == k


def test_gate_accepts_target_argmax():
    g = np.random.default_rng(2)
    V, k = 40, 3
    zd = _rows(g, V, k, 0.0)
    zt = _rows(g, V, k + 1, 0.0)
    ys = [int(np.argmax(z)) for z in zt[:k]]
    res = O.verify_sequence(zt, zd, ys, [1.0 - 2.0 ** -24] * (k + 1), [1.0] * k, k, O.MODE_CM, 1, 0.0, 0.0)
    assert all(p["gate"] for p in res["positions"])
    assert res["n_acc"] == k


def test_degenerate_equal_rows_and_masked_draft():
    g = np.random.default_rng(4)
    V, k = 30, 4
    zd = _rows(g, V, k, 0.0)
    zt = [z.copy() for z in zd] + _rows(g, V, 1, 0.0)
    ys = [int(v) for v in g.integers(0, V, k)]
    for mode in (O.MODE_STANDARD, O.MODE_CM):
        res = O.verify_sequence(zt, zd, ys, [1.0 - 2.0 ** -24] * (k + 1), [0.2] * k, k, mode, 3, 0.1, 1.0)
        assert res["n_acc"] == k           # p_t = p_d: every draft accepted
    zt2 = [z.copy() for z in zt]
    zt2[1][ys[1]] = -math.inf               # target gives the drafted token zero mass
    for mode in (O.MODE_STANDARD, O.MODE_CM):
        res = O.verify_sequence(zt2, zd, ys, [0.0] * (k + 1), [1.0] * k, k, mode, V, 1e9, 0.0)
        assert not res["flags"][1]
        assert res["n_acc"] == 1
        assert zt2[1][res["next"]] > -math.inf


def test_final_sample_uses_rejection_row_or_bonus_row():
    V, k = 6, 2
    zd = [np.log(np.array([0.5, 0.5, 1e-300, 1e-300, 1e-300, 1e-300])), np.zeros(V)]
    zt = [np.log(np.array([0.5, 0.0 + 1e-300, 0.5, 1e-300, 1e-300, 1e-300])), np.zeros(V),
          np.array([-math.inf] * 5 + [0.0])]
    # draft token 1 at position 0 has p_t ~ 0: rejected; residual max(0, p_t - p_d) puts
    # all mass on token 2
    res = O.verify_sequence(zt, zd, [1, 0], [0.5, 0.5, 0.77], [0.5, 0.5], k, O.MODE_STANDARD, 3, 0.1, 1.0)
    assert res["n_acc"] == 0 and res["next"] == 2
    # equal rows at position 1 and an accepted position 0: bonus token from target row k = 2
    res = O.verify_sequence(zt, zd, [0, 3], [0.0, 0.0, 0.3], [0.5, 0.5], k, O.MODE_STANDARD, 3, 0.1, 1.0)
    assert res["n_acc"] == 2 and res["next"] == 5


def test_zero_residual_falls_back_to_the_rejecting_rows_target():
    # Drafter and target rows are equal at both positions, and the draft at position 1
    # is a token that both rows mask (z = -inf): p_t(y) = 0 rejects it with certainty,
    # and the residual max(0, p_t - p_d) of two equal rows is identically zero, so the
    # final token comes from the fallback, p_t of that same row (reading R13).
    #   row 1 = [0, ln 2, -inf, 0]: p = [1/4, 1/2, 0, 1/4], CDF = [1/4, 3/4, 3/4, 1]
    #   inverse CDF (smallest y with CDF(y) > u): u = 0.1 -> 0, u = 0.5 -> 1,
    #   u = 0.8 -> 3 (the masked token 2 adds no mass and is never returned).
    # The bonus row [ln 8, 0, 0, 0] (p = [8, 1, 1, 1]/11, CDF 8/11, 9/11, 10/11, 1)
    # would give 0, 0 and 1 instead, and a uniform fallback 0, 2 and 3.
    r0 = np.array([0.0, 1.0, -0.5, 0.25])
    r1 = np.array([0.0, math.log(2.0), -math.inf, 0.0])
    bonus = np.array([math.log(8.0), 0.0, 0.0, 0.0])
    zd = [r0, r1]
    zt = [r0.copy(), r1.copy(), bonus]
    ys = [1, 2]            # position 0: equal rows, accepted for any u < 1; position 1: masked
    rs1 = O.row_stats(r1)
    q = O.residual_pmf(r1, rs1, r1, rs1)
    assert np.all(np.abs(q - np.array([0.25, 0.5, 0.0, 0.25])) <= 1e-15)
    for mode in (O.MODE_STANDARD, O.MODE_CM):
        for u, want in ((0.1, 0), (0.5, 1), (0.8, 3)):
            res = O.verify_sequence(zt, zd, ys, [0.3, 0.3, u], [0.9, 0.9], 2, mode, 3, 0.1, 1.0)
            assert res["flags"] == [True, False]
            assert res["n_acc"] == 1
            assert res["next"] == want, (mode, u, res["next"])
    # GREEDY takes the top token of the rejecting row instead of sampling: index 1
    res = O.verify_sequence(zt, zd, ys, [0.3, 0.3, 0.8], [0.9, 0.9], 2, O.MODE_GREEDY, 3, 0.1, 1.0)
    assert res["n_acc"] == 1 and res["next"] == 1


# ----------------------------------------------------------------------------- GREEDY mode
@pytest.mark.parametrize("seed", range(12))
def test_greedy_exact_match_reduction(seed):
    # beta = 1, tau_t = 0: the accepted prefix is the longest run of drafts equal to
    # the target's top token, and the next token is the target's top token right after
    # (Sec. III.A step 2), written here as a direct scan
    g = np.random.default_rng(300 + seed)
    V, k = int(g.integers(2, 7)), int(g.integers(1, 6))
    zt = [g.integers(-2, 3, V).astype(np.float64) for _ in range(k + 1)]
    zd = _rows(g, V, k, 0.0)
    ys = [int(v) for v in g.integers(0, V, k)]
    for i in range(k):                      # make some drafts hit the top token
        if g.random() < 0.6:
            ys[i] = int(np.argmax(zt[i]))
    res = O.verify_sequence(zt, zd, ys, [0.5] * (k + 1), [0.3] * k, k, O.MODE_GREEDY, 1, 0.0, 0.0)
    c = 0
    while c < k and zt[c][ys[c]] == zt[c].max():
        c += 1
    top = max(range(V), key=lambda v: (zt[c][v], -v))
    assert res["n_acc"] == c
    assert res["next"] == top


@pytest.mark.parametrize("seed", range(12))
def test_greedy_without_gate_is_exact_match(seed):
    # beta = 0 turns the gate off: a draft passes only as the target's top token, the
    # lowest index among equal maxima (tied maxima at higher indices are rejected),
    # whatever tau; written here as a direct scan
    g = np.random.default_rng(500 + seed)
    V, k = int(g.integers(2, 7)), int(g.integers(1, 6))
    zt = [g.integers(-2, 3, V).astype(np.float64) for _ in range(k + 1)]
    zd = _rows(g, V, k, 0.0)
    ys = [int(v) for v in g.integers(0, V, k)]
    for i in range(k):
        if g.random() < 0.6:
            ys[i] = int(np.flatnonzero(zt[i] == zt[i].max())[-1])   # the last tied max
        if g.random() < 0.5:
            ys[i] = int(np.flatnonzero(zt[i] == zt[i].max())[0])
    res = O.verify_sequence(zt, zd, ys, [0.5] * (k + 1), [0.3] * k, k, O.MODE_GREEDY, 0, 5.0, 1.0)
    c = 0
    while c < k and ys[c] == min(v for v in range(V) if zt[c][v] == zt[c].max()):
        c += 1
    assert res["n_acc"] == c
    assert res["next"] == min(v for v in range(V) if zt[c][v] == zt[c].max())


def test_greedy_accepts_every_exact_match():
    # the target's top token passes for any gate setting, even a negative threshold
    g = np.random.default_rng(12)
    V, k = 40, 6
    for _ in range(20):
        zd = _rows(g, V, k, 0.0)
        zt = _rows(g, V, k + 1, 0.0)
        ys = [int(np.argmax(zt[i])) for i in range(k)]
        for beta, tau, gamma in ((0, 0.0, 0.0), (1, -1.0, 0.0), (3, 0.1, -5.0), (V, 100.0, 1.0)):
            assert O.verify_sequence(zt, zd, ys, [0.0] * (k + 1), [0.5] * k, k, O.MODE_GREEDY, beta, tau,
                                     gamma)["n_acc"] == k


def test_greedy_gate_monotone_in_beta_and_tau():
    g = np.random.default_rng(11)
    V, k = 30, 5
    for _ in range(30):
        zd = _rows(g, V, k, 0.0)
        zt = _rows(g, V, k + 1, 0.0)
        ys = [int(v) for v in g.integers(0, V, k)]
        C = g.random(k).tolist()
        prev = -1
        for beta, tau in ((1, 0.0), (2, 0.5), (5, 1.0), (V, 100.0)):
            n = O.verify_sequence(zt, zd, ys, [0.0] * (k + 1), C, k, O.MODE_GREEDY, beta, tau, 0.0)["n_acc"]
            assert n >= prev
            prev = n
        assert prev == k                     # everything passes a gate of top-|V| and a huge tau


@pytest.mark.parametrize("seed", range(5))
def test_draft_sample_exact_measure(seed):
    # over the 2^24-point uniform lattice, token y is drawn with probability p_d(y)
    g = np.random.default_rng(500 + seed)
    V = int(g.integers(2, 9))
    z = _rows(g, V, 1, 0.25)[0]
    p = softmax(z)
    starts = [first_true(lambda j, y=y: O.draft_sample(z, u_at(j))[0] >= y) for y in range(V)] + [N]
    for y in range(V):
        assert (starts[y + 1] - starts[y]) / N == pytest.approx(p[y], abs=2.0 / N)
