"""The GPU path, through the C ABI, against the hand-worked example in
tests/golden/worked_example.json (closed forms from Sec. III.B(1), III.B(b),
III.B(c) and standard speculative sampling): drafter stats, draft lengths, and
every verification case by cmsd_verify and by cmsd_logit_pass."""
import math

import numpy as np
import pytest
import torch

from tests import golden_example as G
from tests import harness as Hn

pytestmark = pytest.mark.gpu
FX = G.load()


@pytest.fixture(scope="module")
def cm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_15371_amd import cmsd
    return cmsd


def _dev(rows):
    return torch.tensor(np.array(rows, dtype=np.float32), device="cuda:0")


def _close(gpu, ref):
    # fp32 inputs and fp32 outputs of closed forms that are O(1)
    if math.isinf(ref):
        return gpu == ref
    return abs(gpu - ref) <= 2e-6 * max(1.0, abs(ref))


def test_drafter_stats(cm):
    st = cm.cmsd_confidence(_dev(FX["drafter_z"]), lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin=1.0)
    g = Hn.stats_np(st)
    for r, row in enumerate(FX["drafter_rows"]):
        assert _close(float(g["H"][r]), G.value(row["H"])), (r, g["H"][r])
        assert _close(float(g["msoft"][r]), G.value(row["margin_soft"])), r
        assert _close(float(g["mlogit"][r]), G.value(row["margin_logit"])), r
        assert _close(float(g["C"][r]), G.value(row["C"])), (r, g["C"][r])
        assert int(g["top1"][r]) == row["top1"]


@pytest.mark.parametrize("case", FX["draft_len"], ids=lambda c: f"alpha{c['alpha']}-kmin{c['k_min']}")
def test_draft_length(cm, case):
    st = cm.cmsd_confidence(_dev(FX["drafter_z"]), lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin=1.0)
    k, off = cm.cmsd_draft_len(st, 1, k_min=case["k_min"], k_max=4, alpha=case["alpha"])
    assert k.cpu().tolist() == [case["k"]]
    assert off.cpu().tolist() == [0, case["k"] + 1]


def _inputs(cm, case):
    dev = torch.device("cuda:0")
    draft = _dev(FX["drafter_z"])
    drafted = torch.tensor(FX["verify"]["drafted"] + [0, 0], dtype=torch.int32, device=dev)
    st = cm.cmsd_confidence(draft, lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin=1.0)
    kw = dict(mode=G.MODES[case["mode"]], top_beta=case.get("top_beta", 3), tau_base=0.1,
              gamma=case.get("gamma", 1.0))
    return draft, drafted, st, kw


@pytest.mark.parametrize("case", FX["verify"]["cases"], ids=lambda c: f"{c['mode']}-{c['u']}-{c.get('gamma', 1)}-"
                                                                   f"{c.get('top_beta', 3)}")
def test_verify(cm, case):
    dev = torch.device("cuda:0")
    draft, drafted, st, kw = _inputs(cm, case)
    k, off = cm.cmsd_draft_len(st, 1, k_min=1, k_max=4, alpha=1.0)   # k_b = 2
    target = _dev(FX["target_z"])                                      # rows t0, t1, t2 packed
    unif = torch.tensor(case["u"], dtype=torch.float32, device=dev)
    n_acc, nxt, _ = cm.cmsd_verify(draft, st, target, off, k, drafted, unif, batch=1, k_max=4, **kw)
    assert (int(n_acc.item()), int(nxt.item())) == (case["n_acc"], case["next"])


@pytest.mark.parametrize("case", FX["verify"]["cases"], ids=lambda c: f"{c['mode']}-{c['u']}-{c.get('gamma', 1)}-"
                                                                   f"{c.get('top_beta', 3)}")
def test_logit_pass_adaptive(cm, case):
    # the dense layout holds k_max + 1 = 5 target rows; verifying the first k_b = 2
    # drafts makes row 2 (t2) the final row, rows 3 and 4 are never used
    dev = torch.device("cuda:0")
    draft, drafted, _, kw = _inputs(cm, case)
    tz = FX["target_z"]
    target = _dev(tz + [tz[2], tz[2]])
    unif = torch.tensor(case["u"] + [0.0, 0.0], dtype=torch.float32, device=dev)
    out = cm.cmsd_logit_pass(draft, target, drafted, unif, batch=1, k_max=4, lambdas=(1 / 3, 1 / 3, 1 / 3),
                             beta_margin=1.0, k_min=1, alpha=1.0, adaptive=True, **kw)
    torch.cuda.synchronize()
    assert int(out["draft_len"].item()) == 2
    assert (int(out["n_accepted"].item()), int(out["next_token"].item())) == (case["n_acc"], case["next"])
