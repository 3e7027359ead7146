"""Table III ablation settings as parameter presets (host logic only)."""
import pytest

pipeline = pytest.importorskip("paper_2508_15371_amd.pipeline")


def test_presets():
    p = pipeline.Params()
    assert p.fixed_k(16).k_min == 16 and p.fixed_k(16).gamma == p.gamma
    assert p.fixed_tau().gamma == 0.0 and p.fixed_tau().k_min == p.k_min
    q = p.fixed_k_and_tau(8)
    assert q.k_min == 8 and q.gamma == 0.0
    assert p.entropy_only().lambdas == (1.0, 0.0, 0.0)
    assert p.margin_only().lambdas == (0.0, 1.0, 0.0)
    assert p.softmax_only().lambdas == (0.0, 0.0, 1.0)
    assert p.lambdas == (1 / 3, 1 / 3, 1 / 3)          # presets copy, never mutate
