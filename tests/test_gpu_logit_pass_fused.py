"""GPU parity of cmsd_logit_pass_fused, the one-launch logit pass for small batches
(Sec. III.B(1)-(c), Sec. III.A): bit-equal to cmsd_logit_pass (the same arithmetic in
one launch), checked against the oracle, repeated calls on one workspace (its
per-sequence counters return to zero), invalid ids, and HIP graph replays."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import cmsd_oracle as O
from tests import harness as Hn
from tests.test_gpu_logit_pass import _case, _check

pytestmark = pytest.mark.gpu

FIELDS = ("draft_stats", "draft_len", "target_stats", "n_accepted", "next_token")


@pytest.fixture(autouse=True)
def _row_block_256(row_shape):
    # the fused pass runs its rows with 256 threads; the four-launch pass it is compared
    # with bit for bit must too, also when a run forces another size for every launch
    row_shape(256)


@pytest.fixture(scope="module")
def cm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_15371_amd import cmsd
    return cmsd


def _kw(mode, adaptive, **over):
    P = dict(Hn.PARAMS)
    P.update(over)
    return P, dict(lambdas=P["lambdas"], beta_margin=P["beta_margin"], k_min=P["k_min"], alpha=P["alpha"],
                   mode=mode, top_beta=P["top_beta"], tau_base=P["tau_base"], gamma=P["gamma"], adaptive=adaptive)


def _both(cm, dd, td, dr, u, B, K, mode, adaptive, ws=None, **over):
    """The four-launch pass and the fused one on the same inputs."""
    P, kw = _kw(mode, adaptive, **over)
    uu = None if mode == O.MODE_GREEDY else u
    ref = cm.cmsd_logit_pass(dd, td, dr, uu, batch=B, k_max=K, **kw)
    fus = cm.cmsd_logit_pass_fused(dd, td, dr, uu, batch=B, k_max=K, workspace=ws, **kw)
    torch.cuda.synchronize()
    return ref, fus, P


def _assert_equal(ref, fus, tag=""):
    for f in FIELDS:
        assert torch.equal(ref[f].view(torch.int32), fus[f].view(torch.int32)), (tag, f)


def _counters(ws, B):
    # the per-sequence counters end the workspace
    end = (ws.numel() * ws.element_size()) & ~3
    return ws.view(torch.uint8)[end - 4 * B:end].view(torch.int32)


@pytest.mark.parametrize("adaptive", [False, True])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
@pytest.mark.parametrize("name", ["tiny", "b1", "c2"])
def test_fused_equals_logit_pass_and_oracle(cm, name, mode, adaptive):
    print(f"[fused parity] start {name} mode={mode} adaptive={adaptive}", flush=True)
    cfg = W.CONFIGS[name]
    d = Hn.workload(name)
    ref, fus, P = _both(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max,
                        mode, adaptive)
    _assert_equal(ref, fus, name)
    t = Hn.Tally()
    n_acc, k = _check(t, cfg.B, cfg.k_max, cfg.V, cfg.dtype, d["draft"], d["target"], d["drafted"], d["uniforms"],
                      fus, P, mode, adaptive, list(range(cfg.B)))
    print(f"[fused parity] {name} mode={mode} adaptive={adaptive}: checked={t.checked} exceptions={t.exceptions} "
          f"mean n_acc={n_acc.mean():.3f}", flush=True)
    t.assert_ok()
    assert int(_counters(fus["workspace"], cfg.B).abs().sum()) == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V,K,B,pad", [(2, 1, 3, 0), (37, 3, 5, 3), (1000, 63, 2, 0), (4099, 5, 4, 5),
                                       (50257, 7, 3, 1), (300007, 2, 2, 0)])
def test_fused_shapes(cm, dtype, V, K, B, pad):
    g = np.random.default_rng(V * 11 + K)
    zd, zt, dr, u = _case(g, B, K, V, dtype)
    dev = torch.device("cuda:0")
    dd = Hn.to_device(zd, dtype, dev)
    td = Hn.to_device(zt, dtype, dev)
    if pad:
        dd = torch.nn.functional.pad(dd, (0, pad))[:, :V]
        td = torch.nn.functional.pad(td, (0, pad))[:, :V]
    drd = torch.from_numpy(dr.reshape(-1)).to(dev)
    ud = torch.from_numpy(u.reshape(-1)).to(dev)
    ws = cm.fused_workspace(B, K, V, dev)
    for mode in (O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY):
        adaptive = mode == O.MODE_CM
        ref, fus, P = _both(cm, dd, td, drd, ud, B, K, mode, adaptive, ws=ws)
        _assert_equal(ref, fus, (V, K, B, mode))
        t = Hn.Tally()
        _check(t, B, K, V, dtype, zd, zt, dr, u, fus, P, mode, adaptive, list(range(B)))
        t.assert_ok()
    assert int(_counters(ws, B).abs().sum()) == 0


def test_fused_repeated_calls_one_workspace(cm):
    # successive calls on one workspace, on different inputs and batch sizes up to its
    # own: each matches the four-launch pass, and the counters end at zero every time
    V, K, B = 3001, 6, 7
    dev = torch.device("cuda:0")
    ws = cm.fused_workspace(B, K, V, dev)
    for rep, b in enumerate((7, 7, 3, 7, 1)):
        g = np.random.default_rng(40 + rep)
        zd, zt, dr, u = _case(g, b, K, V, "bf16")
        ref, fus, _ = _both(cm, Hn.to_device(zd, "bf16", dev), Hn.to_device(zt, "bf16", dev),
                            torch.from_numpy(dr.reshape(-1)).to(dev), torch.from_numpy(u.reshape(-1)).to(dev),
                            b, K, O.MODE_CM, True, ws=ws)
        _assert_equal(ref, fus, rep)
        assert int(_counters(ws, B).abs().sum()) == 0, rep


def test_fused_invalid_drafted_id(cm):
    V, K, B = 500, 4, 3
    g = np.random.default_rng(8)
    zd, zt, dr, u = _case(g, B, K, V, "f32")
    dr[1, 3] = V          # out of range: sequence 1 is invalid, the others are not
    dev = torch.device("cuda:0")
    for mode in (O.MODE_CM, O.MODE_GREEDY):
        ref, fus, _ = _both(cm, Hn.to_device(zd, "f32", dev), Hn.to_device(zt, "f32", dev),
                            torch.from_numpy(dr.reshape(-1)).to(dev), torch.from_numpy(u.reshape(-1)).to(dev),
                            B, K, mode, False)
        _assert_equal(ref, fus, mode)
        n_acc = fus["n_accepted"].cpu().numpy()
        assert n_acc[1] == -1 and int(fus["next_token"][1]) == -1 and n_acc[0] >= 0 and n_acc[2] >= 0


@pytest.mark.parametrize("mode", [O.MODE_CM, O.MODE_GREEDY])
def test_fused_graph_replays_match_eager(cm, mode):
    # a fused call captured in a HIP graph: every replay (eager work in between)
    # matches the eager four-launch pass, and each leaves the counters at zero
    from paper_2508_15371_amd import pipeline
    cfg = W.CONFIGS["c2"]
    d = Hn.workload("c2")
    args = (d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"])
    ref = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", pipeline.Params(mode=mode))
    ref.logit_pass(*args)
    torch.cuda.synchronize()
    fields = ("stats", "k", "tstats", "n_acc", "next_tok")
    want = {f: getattr(ref, f).clone() for f in fields}
    lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", pipeline.Params(mode=mode))
    lp.logit_pass_fused(*args)                     # warm-up (and workspace) outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lp.logit_pass_fused(*args)
    junk = torch.zeros(1 << 20, device="cuda:0")
    for rep in range(4):
        lp.stats.fill_(float("nan"))
        lp.tstats.fill_(float("nan"))
        lp.k.fill_(-7)
        lp.n_acc.fill_(-7)
        lp.next_tok.fill_(-7)
        junk.add_(1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for f in fields:
            assert torch.equal(getattr(lp, f).view(torch.int32), want[f].view(torch.int32)), (rep, f)
        assert int(_counters(lp.fws, cfg.B).abs().sum()) == 0, rep
