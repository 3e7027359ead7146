"""Pins of the oracle's adaptive draft length (Sec. III.B(b)).  CPU only."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import cmsd_oracle as O


def test_exact_grid_against_rationals():
    # confidences on a dyadic grid make alpha*Cbar*k_max exact, so the floor and clip
    # can be checked with exact rational arithmetic
    g = np.random.default_rng(7)
    for k_max in (1, 2, 5, 8, 16):
        for k_min in range(1, k_max + 1):
            for alpha in (1.0, 0.75, 0.5, 0.125):
                B = 40
                num = g.integers(0, 65, size=(B, k_max))
                C = num / 64.0
                k, off, slack = O.draft_len(C, k_min, k_max, alpha)
                for b in range(B):
                    x = Fraction(alpha) * sum(Fraction(int(n), 64) for n in num[b])
                    want = min(k_max, max(k_min, math.floor(x)))
                    assert k[b] == want
                acc = 0
                for b in range(B):
                    assert off[b] == acc
                    acc += int(k[b]) + 1
                assert off[B] == acc


def test_full_confidence_gives_k_max_and_fixed_k():
    C = np.ones((3, 16))
    k, _, _ = O.draft_len(C, 1, 16, 1.0)
    assert (k == 16).all()
    # k_min = k_max: a fixed draft length whatever the confidence
    for c in (0.0, 0.3, 1.0):
        k, off, slack = O.draft_len(np.full((4, 8), c), 8, 8, 1.0)
        assert (k == 8).all()
        assert (off == np.arange(5) * 9).all()
        assert np.isinf(slack).all()
    # zero confidence drafts k_min (never zero tokens)
    k, _, _ = O.draft_len(np.zeros((2, 16)), 1, 16, 1.0)
    assert (k == 1).all()


def test_monotone_in_alpha_and_confidence():
    g = np.random.default_rng(3)
    C = g.uniform(0, 1, (200, 16))
    prev = None
    for alpha in np.linspace(0.05, 1.0, 20):
        k, _, _ = O.draft_len(C, 2, 16, float(alpha))
        assert ((k >= 2) & (k <= 16)).all()
        if prev is not None:
            assert (k >= prev).all()
        prev = k
    k1, _, _ = O.draft_len(C, 1, 16, 0.9)
    k2, _, _ = O.draft_len(np.minimum(1.0, C + 0.05), 1, 16, 0.9)
    assert (k2 >= k1).all()


def test_slack_is_distance_to_relevant_integer():
    k_max = 8
    C = np.full((1, k_max), 0.5)          # x = 4 exactly
    _, _, s = O.draft_len(C, 1, k_max, 1.0)
    assert s[0] == 0.0
    C = np.full((1, k_max), 0.55)         # x = 4.4
    _, _, s = O.draft_len(C, 1, k_max, 1.0)
    assert s[0] == pytest.approx(0.4)
    C = np.full((1, k_max), 0.01)         # x = 0.08, nearest 0 is clipped away
    _, _, s = O.draft_len(C, 1, k_max, 1.0)
    assert s[0] == math.inf
