"""cmsd_logit_pass_noalloc, the logit pass on the library's static per-device scratch
(for callers that cannot allocate), against cmsd_logit_pass on a caller workspace:
every output bit-identical, over consecutive calls of different sizes that share the
scratch (the later, smaller call must not see the earlier one's contents)."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import cmsd_oracle as O
from tests import harness as Hn

pytestmark = pytest.mark.gpu

FIELDS = ("draft_stats", "draft_len", "target_stats", "n_accepted", "next_token")


@pytest.fixture(scope="module")
def cm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_15371_amd import cmsd
    return cmsd


def _inputs(seed, B, K, V, dtype):
    g = np.random.default_rng(seed)
    zd = g.normal(0, 2.0, (B * K, V)).astype(np.float32)
    zt = g.normal(0, 2.0, (B * (K + 1), V)).astype(np.float32)
    for b in range(B):
        for i in range(K):
            zt[b * (K + 1) + i] = zd[b * K + i] + g.normal(0, 0.5, V).astype(np.float32)
    store = (lambda x: x) if dtype == "f32" else W.bf16_bits_from_f32
    zd, zt = store(zd), store(zt)
    drafted = np.array([[int(np.argmax(Hn.decode(zd[b * K + i], dtype) + g.gumbel(size=V))) for i in range(K)]
                        for b in range(B)], dtype=np.int32)
    unif = (g.integers(0, 1 << 24, (B, K + 1)) * 2.0 ** -24).astype(np.float32)
    dev = torch.device("cuda:0")
    return (Hn.to_device(zd, dtype, dev), Hn.to_device(zt, dtype, dev),
            torch.from_numpy(drafted.reshape(-1)).to(dev), torch.from_numpy(unif.reshape(-1)).to(dev))


def _outs(B, K, dev):
    return {"draft_stats": torch.empty((B * K, 8), dtype=torch.float32, device=dev),
            "draft_len": torch.empty(B, dtype=torch.int32, device=dev),
            "target_stats": torch.empty((B * (K + 1), 8), dtype=torch.float32, device=dev),
            "n_accepted": torch.empty(B, dtype=torch.int32, device=dev),
            "next_token": torch.empty(B, dtype=torch.int32, device=dev)}


@pytest.mark.parametrize("decisions", [0, 1])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
def test_noalloc_equals_logit_pass_on_consecutive_calls(cm, mode, decisions):
    # decisions: 0 = the per-call choice (formed in the final-token kernels at these
    # sizes), 1 = the decision kernel's record, written over the scratch's row slots
    cm.cmsd_set_pass_decisions(decisions)
    try:
        _consecutive_calls(cm, mode)
    finally:
        cm.cmsd_set_pass_decisions(0)


def _consecutive_calls(cm, mode):
    dev = torch.device("cuda:0")
    # a larger call, then a smaller one of another dtype and vocabulary on the same
    # scratch, then the larger one again
    cases = [(11, 24, 8, 50257, "bf16", False), (12, 5, 4, 3001, "f32", True), (11, 24, 8, 50257, "bf16", False)]
    for seed, B, K, V, dtype, adaptive in cases:
        print(f"[noalloc] mode={mode} B={B} K={K} V={V} {dtype} adaptive={adaptive}", flush=True)
        dd, td, dr, u = _inputs(seed, B, K, V, dtype)
        if mode == O.MODE_GREEDY:
            u = None
        kw = dict(batch=B, k_max=K, mode=mode, adaptive=adaptive, **{k: v for k, v in Hn.PARAMS.items()})
        ref = cm.cmsd_logit_pass(dd, td, dr, u, **kw)
        ref = {k: ref[k].clone() for k in FIELDS}
        outs = _outs(B, K, dev)
        for t in outs.values():
            t.fill_(-7)                  # stale values the call must overwrite
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        got = cm.cmsd_logit_pass_noalloc(dd, td, dr, u, **kw, **outs)
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info()[0] == free0, "the no-allocation call changed free device memory"
        for k in FIELDS:
            assert got[k] is outs[k]
            assert torch.equal(got[k].view(torch.int32), ref[k].view(torch.int32)), (k, B, K, V)
        assert int(got["n_accepted"].min()) >= 0


def test_noalloc_rejects_problems_beyond_the_scratch(cm):
    B, K, V = 4096, 16, 128256              # 18.7 MB of workspace: over the 16 MiB scratch
    assert cm.cmsd_verify_workspace_bytes(B, K, V) > cm.CMSD_STATIC_SCRATCH_BYTES
    # through the raw entry point with fake, aligned addresses: rejected on the host
    import ctypes as C
    P = 0x10000
    st = cm.lib().cmsd_logit_pass_noalloc(P, V, P, V, P, P, cm.CMSD_BF16, B, K, V,
                                          C.byref(cm.ConfParams(1 / 3, 1 / 3, 1 / 3, 1.0)),
                                          C.byref(cm.DraftParams(1, K, 1.0)),
                                          C.byref(cm.VerifyParams(1, 3, 0.1, 1.0)), 0, P, P, P, P, P, None)
    assert st == cm.CMSD_ERR_SIZE
