"""The Python binding rejects caller buffers of the wrong dtype, layout or size
before any device work (the C entry points take plain pointers and cannot check
sizes).  CPU only: the checks run on tensor metadata."""
import pytest
import torch

cm = pytest.importorskip("paper_2508_15371_amd.cmsd")


def _f(*shape):
    return torch.zeros(*shape, dtype=torch.float32)


def _i(*shape):
    return torch.zeros(*shape, dtype=torch.int32)


def test_confidence_stats_buffer():
    x = _f(4, 100)
    with pytest.raises(ValueError, match="device"):
        cm.cmsd_confidence(x, _f(4, 8))           # sizes fine: only the device check fails
    with pytest.raises(ValueError, match="stats"):
        cm._buf(_f(3, 8), "stats", torch.float32, 32, x.device)
    with pytest.raises(ValueError, match="stats"):
        cm._buf(_f(8, 4).t(), "stats", torch.float32, 32, x.device)   # not contiguous
    with pytest.raises(ValueError, match="stats"):
        cm._buf(_i(4, 8), "stats", torch.float32, 32, x.device)
    cm._buf(_f(4, 8), "stats", torch.float32, 32, x.device)


def test_draft_len_buffers():
    with pytest.raises(ValueError, match="stats"):
        cm.cmsd_draft_len(_f(10, 8), 3, k_min=1, k_max=4, alpha=1.0, draft_len=_i(3), target_offsets=_i(4))
    with pytest.raises(ValueError, match="draft_len"):
        cm.cmsd_draft_len(_f(12, 8), 3, k_min=1, k_max=4, alpha=1.0, draft_len=_i(2), target_offsets=_i(4))
    with pytest.raises(ValueError, match="target_offsets"):
        cm.cmsd_draft_len(_f(12, 8), 3, k_min=1, k_max=4, alpha=1.0, draft_len=_i(3), target_offsets=_i(3))


def _verify(**kw):
    B, K, V, R = 3, 4, 50, 15
    a = dict(draft_logits=_f(B * K, V), draft_stats=_f(B * K, 8), target_logits=_f(R, V),
             target_offsets=_i(B + 1), draft_len=_i(B), drafted=_i(B * K), uniforms=_f(R),
             target_stats=_f(R, 8), n_accepted=_i(B), next_token=_i(B),
             workspace=torch.zeros(10000, dtype=torch.float64))
    a.update(kw)
    return cm.cmsd_verify(a.pop("draft_logits"), a.pop("draft_stats"), a.pop("target_logits"),
                          a.pop("target_offsets"), a.pop("draft_len"), a.pop("drafted"), a.pop("uniforms"),
                          batch=B, k_max=K, **a)


@pytest.mark.parametrize("name,bad", [
    ("draft_logits", _f(11, 50)), ("draft_stats", _f(11, 8)), ("target_offsets", _i(3)),
    ("draft_len", _i(2)), ("drafted", _i(11)), ("uniforms", _f(14)), ("target_stats", _f(14, 8)),
    ("n_accepted", _i(2)), ("next_token", _i(2)), ("drafted", torch.zeros(12, dtype=torch.int64)),
    ("workspace", torch.zeros(10000, dtype=torch.float32)),
])
def test_verify_buffers(name, bad):
    with pytest.raises(ValueError, match=name):
        _verify(**{name: bad})


def test_verify_sizes_ok_reach_device_check():
    with pytest.raises(ValueError, match="device"):
        _verify()


def test_draft_sample_buffers():
    x = _f(5, 70)
    with pytest.raises(ValueError, match="device"):
        cm.cmsd_draft_sample(x, _f(5, 8), _f(5), drafted=_i(5), workspace=torch.zeros(100, dtype=torch.float64))
