"""Pins of the oracle's per-row statistics and confidence (Sec. III.B(1)) against
closed forms, a library cross-check, brute force and invariances.  CPU only."""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import cmsd_oracle as O


def _rng(s):
    return np.random.default_rng(1234 + s)


@pytest.mark.parametrize("V", [2, 3, 1024, 32000, 128256])
def test_uniform_row_has_max_entropy(V):
    # a uniform distribution has entropy log|V|, the maximum (Sec. III.B(1)); no margin
    z = np.full(V, 0.37)
    rs = O.row_stats(z)
    assert rs.H == pytest.approx(math.log(V), rel=1e-13, abs=1e-13)
    assert rs.p1_minus_p2 == 0.0
    assert rs.margin_logit == 0.0
    assert rs.top1 == 0
    c_ent, c_m, c_s = O.normalised_signals(rs, V, 1.0)
    assert c_ent == pytest.approx(0.0, abs=1e-13)
    assert c_m == 0.5
    assert c_s == 0.0


@pytest.mark.parametrize("V,hot", [(8, 3), (1024, 0), (50257, 50256)])
@pytest.mark.parametrize("fill", [-math.inf, -800.0])
def test_one_hot_row(V, hot, fill):
    # a one-hot distribution: zero entropy, softmax margin 1, full confidence
    z = np.full(V, fill)
    z[hot] = 0.0 if fill == -math.inf else 5.0
    rs = O.row_stats(z)
    assert rs.H == 0.0
    assert rs.top1 == hot
    assert rs.p1_minus_p2 == 1.0
    c_ent, c_m, c_s = O.normalised_signals(rs, V, 1.0)
    assert c_ent == 1.0 and c_s == 1.0
    assert c_m == 1.0 if fill == -math.inf else c_m == pytest.approx(1.0)
    assert O.confidence(rs, V, (1 / 3, 1 / 3, 1 / 3), 1.0) == pytest.approx(1.0)


@pytest.mark.parametrize("delta", [0.0, 1e-3, 0.5, 2.0, 7.5, 30.0])
def test_two_point_row_closed_form(delta):
    # two finite logits: softmax is (sigmoid(d), 1 - sigmoid(d)); entropy is the
    # binary entropy and the softmax margin is tanh(d/2)
    V = 16
    z = np.full(V, -math.inf)
    z[5] = 1.25 + delta
    z[11] = 1.25
    rs = O.row_stats(z)
    p = 1.0 / (1.0 + math.exp(-delta))      # sigmoid(d)
    q = 1.0 / (1.0 + math.exp(delta))       # 1 - sigmoid(d), without cancellation
    h = p * math.log1p(math.exp(-delta)) + q * math.log1p(math.exp(delta))
    assert rs.H == pytest.approx(h, rel=1e-12, abs=1e-15)
    assert rs.p1_minus_p2 == pytest.approx(math.tanh(delta / 2), rel=1e-12, abs=1e-15)
    assert rs.margin_logit == pytest.approx(delta, abs=1e-15)
    assert rs.top1 == (5 if delta > 0 else 5)  # tie at delta=0 -> lowest index 5


@pytest.mark.parametrize("seed", range(6))
def test_entropy_matches_scipy(seed):
    g = _rng(seed)
    V = int(g.integers(2, 5000))
    z = g.normal(0, float(g.uniform(0.1, 10)), V)
    rs = O.row_stats(z)
    p = scipy.special.softmax(z)
    assert rs.H == pytest.approx(float(scipy.stats.entropy(p)), rel=1e-10, abs=1e-14)
    srt = np.sort(p)[::-1]
    assert rs.p1_minus_p2 == pytest.approx(float(srt[0] - srt[1]), rel=1e-10, abs=1e-15)
    assert rs.A * math.exp(rs.m) == pytest.approx(float(np.exp(z).sum()), rel=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_shift_and_permutation_invariance(seed):
    g = _rng(seed)
    V = 777
    z = g.normal(0, 3, V)
    rs = O.row_stats(z)
    rs_s = O.row_stats(z + 12.5)
    assert rs_s.H == pytest.approx(rs.H, rel=1e-12)
    assert rs_s.p1_minus_p2 == pytest.approx(rs.p1_minus_p2, rel=1e-12)
    assert rs_s.margin_logit == pytest.approx(rs.margin_logit, rel=1e-9)
    perm = g.permutation(V)
    rs_p = O.row_stats(z[perm])
    assert rs_p.H == pytest.approx(rs.H, rel=1e-12)
    assert rs_p.p1_minus_p2 == pytest.approx(rs.p1_minus_p2, rel=1e-12)
    assert rs_p.margin_logit == rs.margin_logit
    assert perm[rs_p.top1] == rs.top1


@pytest.mark.parametrize("seed", range(20))
def test_top1_top2_brute_force(seed):
    # small integer logits force ties; top-1 = lowest index of the max, top-2 = the
    # second element of the descending-sorted multiset
    g = _rng(seed)
    V = int(g.integers(2, 12))
    z = g.integers(-3, 3, V).astype(np.float64)
    if seed % 5 == 0:
        z[g.integers(0, V)] = -math.inf
    rs = O.row_stats(z)
    best = 0
    for v in range(V):
        if z[v] > z[best]:
            best = v
    assert rs.top1 == best
    srt = sorted(z.tolist(), reverse=True)
    assert rs.m == srt[0]
    assert rs.z2 == srt[1]
    assert rs.margin_logit == (srt[0] - srt[1] if srt[1] > -math.inf else math.inf)


@pytest.mark.parametrize("seed", range(10))
def test_bounds_and_single_signal_weights(seed):
    g = _rng(seed)
    V = int(g.integers(2, 3000))
    z = g.normal(0, float(g.uniform(0.01, 20)), V)
    rs = O.row_stats(z)
    assert 0.0 <= rs.H <= math.log(V) + 1e-12
    assert 0.0 <= rs.p1_minus_p2 <= 1.0
    sig = O.normalised_signals(rs, V, 1.0)
    for s in sig:
        assert 0.0 <= s <= 1.0
    assert sig[1] >= 0.5
    # one-hot weights reduce C to each single signal (the single-signal ablation settings)
    for j in range(3):
        lam = [0.0, 0.0, 0.0]
        lam[j] = 1.0
        assert O.confidence(rs, V, tuple(lam), 1.0) == sig[j]
    lam = tuple(g.dirichlet([1, 1, 1]))
    C = O.confidence(rs, V, lam, 1.0)
    assert lam[1] / 2 - 1e-12 <= C <= 1.0 + 1e-12


def test_margin_sigmoid_values():
    z = np.array([0.0, -2.0, -5.0, -math.inf])
    rs = O.row_stats(z)
    for bm in (0.25, 1.0, 3.0):
        _, c_m, _ = O.normalised_signals(rs, 4, bm)
        assert c_m == pytest.approx(1 / (1 + math.exp(-2.0 * bm)), rel=1e-15)


def test_decode_logits_bf16():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x7F7F, 0xFF80, 0x3E00], dtype=np.uint16)
    v = O.decode_logits(bits, "bf16")
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 0.0
    assert v[3] == pytest.approx(3.3895313892515355e38)
    assert v[4] == -math.inf
    assert v[5] == 0.125


# ----------------------------------------------------------------------------- logit variance (Sec. I)
@pytest.mark.parametrize("V", [1, 2, 1000])
def test_logit_variance_constant_rows(V):
    assert O.logit_variance(np.full(V, 3.25)) == 0.0
    z = np.full(V + 5, -math.inf)
    z[2] = 7.0                                    # one finite logit
    assert O.logit_variance(z) == 0.0


@pytest.mark.parametrize("n1,n2,a,b", [(1, 1, 0.0, 1.0), (3, 7, -2.5, 4.0), (1, 999, 10.0, 0.0), (500, 500, 1.0, -1.0)])
def test_logit_variance_two_point_closed_form(n1, n2, a, b):
    # n1 logits at a, n2 at b: variance n1 n2 (a - b)^2 / (n1 + n2)^2
    z = np.concatenate([np.full(n1, a), np.full(n2, b), np.full(4, -math.inf)])
    _rng(0).shuffle(z)
    want = n1 * n2 * (a - b) ** 2 / (n1 + n2) ** 2
    assert O.logit_variance(z) == pytest.approx(want, rel=1e-13, abs=1e-15)


@pytest.mark.parametrize("seed", range(8))
def test_logit_variance_pairwise_identity(seed):
    # brute force over pairs: var = sum_i sum_j (z_i - z_j)^2 / (2 n^2), -inf left out
    g = _rng(40 + seed)
    V = int(g.integers(2, 60))
    z = g.normal(0, float(g.uniform(0.1, 20)), V)
    z[g.random(V) < 0.2] = -math.inf
    if not np.isfinite(z).any():
        z[0] = 1.0
    f = z[np.isfinite(z)]
    n = f.size
    want = sum((x - y) ** 2 for x in f for y in f) / (2 * n * n)
    assert O.logit_variance(z) == pytest.approx(want, rel=1e-12, abs=1e-14)


@pytest.mark.parametrize("seed", range(4))
def test_logit_variance_shift_and_scale(seed):
    g = _rng(60 + seed)
    z = g.normal(0, 3, 777)
    v = O.logit_variance(z)
    assert O.logit_variance(z + 1000.0) == pytest.approx(v, rel=1e-9)
    assert O.logit_variance(2.0 * z) == pytest.approx(4.0 * v, rel=1e-13)
    assert O.logit_variance(g.permutation(z)) == pytest.approx(v, rel=1e-13)
