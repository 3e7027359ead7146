"""The oracle against the hand-worked example in tests/golden/worked_example.json
(closed forms derived from Sec. III.B(1), Sec. III.B(b), Sec. III.B(c) and standard
speculative sampling, each with its derivation in the fixture)."""
import math

import numpy as np
import pytest

from oracle import cmsd_oracle as O
from tests import golden_example as G

FX = G.load()
LAM = (1 / 3, 1 / 3, 1 / 3)


def test_expression_evaluator():
    assert G.value("ln(4)") == pytest.approx(2 * math.log(2), abs=1e-15)
    assert G.value("((1 - 0.5/ln(4)) + 3/4)/3") == pytest.approx(((1 - 0.5 / math.log(4)) + 0.75) / 3, abs=1e-15)
    assert G.value("-inf") == -math.inf
    with pytest.raises(ValueError):
        G.value("__import__('os')")


@pytest.mark.parametrize("r", range(4))
def test_row_stats_and_confidence(r):
    row = FX["drafter_rows"][r]
    z = np.array(FX["drafter_z"][r])
    rs = O.row_stats(z)
    assert rs.H == pytest.approx(G.value(row["H"]), abs=1e-12)
    assert rs.p1_minus_p2 == pytest.approx(G.value(row["margin_soft"]), abs=1e-12)
    assert rs.margin_logit == pytest.approx(G.value(row["margin_logit"]), abs=1e-12)
    assert rs.top1 == row["top1"]
    assert O.confidence(rs, FX["vocab"], LAM, 1.0) == pytest.approx(G.value(row["C"]), abs=1e-12)


@pytest.mark.parametrize("case", FX["draft_len"])
def test_draft_length(case):
    C = np.array([[G.value(r["C"]) for r in FX["drafter_rows"]]])
    k, off, _ = O.draft_len(C, case["k_min"], 4, case["alpha"])
    assert int(k[0]) == case["k"]
    assert off.tolist() == [0, case["k"] + 1]


@pytest.mark.parametrize("case", FX["verify"]["cases"], ids=lambda c: f"{c['mode']}-{c['u']}-{c.get('gamma', 1)}")
def test_verify(case):
    zt = [np.array(z) for z in FX["target_z"]]
    zd = [np.array(z) for z in FX["drafter_z"][:2]]
    C = [G.value(r["C"]) for r in FX["drafter_rows"][:2]]
    res = O.verify_sequence(zt, zd, FX["verify"]["drafted"], case["u"], C, 2, G.MODES[case["mode"]],
                            case.get("top_beta", 3), 0.1, case.get("gamma", 1.0))
    assert res["n_acc"] == case["n_acc"]
    assert res["next"] == case["next"]
    # every decision of the example is far from its boundary
    for p in res["positions"]:
        assert min(p["slack_stoch"], p["slack_gap"]) > 0.03
    assert res["slack_next"] > 0.03
