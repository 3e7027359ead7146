"""GPU parity of cmsd_logit_pass, the one-call logit pass of a dense draft
(Sec. III.B(1)-(c), Sec. III.A), against the oracle through the C ABI: drafter
stats, draft lengths, target-row results, accept tests, prefixes and final tokens,
on the dense workloads, in both verification lengths, and on edge cases."""
import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import cmsd_oracle as O
from tests import harness as Hn

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_15371_amd import cmsd
    return cmsd


def _pass(cm, dd, td, drafted, unif, B, K, mode, adaptive=False, **kw):
    P = dict(Hn.PARAMS)
    P.update(kw)
    out = cm.cmsd_logit_pass(dd, td, drafted, None if mode == O.MODE_GREEDY and unif is None else unif,
                             batch=B, k_max=K, lambdas=P["lambdas"], beta_margin=P["beta_margin"],
                             k_min=P["k_min"], alpha=P["alpha"], mode=mode, top_beta=P["top_beta"],
                             tau_base=P["tau_base"], gamma=P["gamma"], adaptive=adaptive)
    torch.cuda.synchronize()
    return out, P


def _check(t, cfg_B, K, V, dtype, draft, target, drafted, uniforms, out, P, mode, adaptive, seqs, stats_rows=True):
    """draft/target: stored host rows; drafted [B, K]; uniforms [B, K+1]."""
    gs = Hn.stats_np(out["draft_stats"])
    ts = Hn.tstats_np(out["target_stats"])
    k_gpu = out["draft_len"].cpu().numpy()
    n_acc = out["n_accepted"].cpu().numpy()
    nxt = out["next_token"].cpu().numpy()
    lam = tuple(Hn.f32(x) for x in P["lambdas"])
    # draft length from the GPU's confidences (stage isolation): bit-exact
    Cg = gs["C"].astype(np.float64).reshape(cfg_B, K)
    k_o, _, _ = O.draft_len(Cg, P["k_min"], K, Hn.f32(P["alpha"]))
    t.value("k(stage)", np.array_equal(k_o, k_gpu), (k_o[:8], k_gpu[:8]))
    for b in seqs:
        zd = [Hn.decode(draft[b * K + i], dtype) for i in range(K)]
        if stats_rows:
            for i in range(K):
                Hn.check_row_stats(t, gs, b * K + i, zd[i], V, lam, Hn.f32(P["beta_margin"]))
        C = [O.confidence(O.row_stats(z), V, lam, Hn.f32(P["beta_margin"])) for z in zd]
        kb_o, _, sl = O.draft_len(np.array([C]), P["k_min"], K, Hn.f32(P["alpha"]))
        t.decision(f"k[{b}]", int(k_gpu[b]), int(kb_o[0]), float(sl[0]))
        kv = int(k_gpu[b]) if adaptive else K
        pos = list(range(kv + 1))
        zt = [Hn.decode(target[b * (K + 1) + i], dtype) for i in pos]
        unif = [float(uniforms[b, i]) for i in pos]
        Hn.check_sequence(t, b, zt, zd, drafted[b], unif, C, kv, mode, P, ts, b * (K + 1), int(n_acc[b]),
                          int(nxt[b]))
    return n_acc, k_gpu


def _seqs(B, n, salt):
    if B <= n:
        return list(range(B))
    g = np.random.default_rng(300 + salt)
    return sorted(set([0, B - 1] + g.choice(B, n, replace=False).tolist()))


@pytest.mark.parametrize("adaptive", [False, True])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
@pytest.mark.parametrize("name,nseq", [("tiny", 1), ("c2", 8), ("c3", 24), ("c4", 3), ("c5", 12), ("v152k", 6)])
def test_logit_pass_configs(cm, name, nseq, mode, adaptive):
    print(f"[logit pass parity] start {name} mode={mode} adaptive={adaptive}", flush=True)
    cfg = W.CONFIGS[name]
    d = Hn.workload(name)
    out, P = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, mode,
                   adaptive)
    t = Hn.Tally()
    seqs = _seqs(cfg.B, nseq, cfg.cid)
    n_acc, k = _check(t, cfg.B, cfg.k_max, cfg.V, cfg.dtype, d["draft"], d["target"], d["drafted"], d["uniforms"],
                      out, P, mode, adaptive, seqs, stats_rows=len(seqs) * cfg.k_max <= 256)
    print(f"[logit pass parity] {name} mode={mode} adaptive={adaptive}: checked={t.checked} "
          f"exceptions={t.exceptions} mean n_acc={n_acc.mean():.3f} mean k={k.mean():.3f}", flush=True)
    t.assert_ok()


@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
def test_bitwise_equal_to_separate_calls(cm, mode):
    # same arithmetic as confidence + draft_len + verify (dense offsets, k = k_max); on
    # c3 both launch their row kernels with 256 threads, so every output is bit-equal
    from paper_2508_15371_amd import pipeline
    cfg = W.CONFIGS["c3"]
    d = Hn.workload("c3")
    out, _ = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, mode)
    lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", pipeline.Params(mode=mode))
    lp.run(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"])
    torch.cuda.synchronize()
    pairs = {"draft_stats": lp.stats, "draft_len": lp.k, "target_stats": lp.tstats, "n_accepted": lp.n_acc,
             "next_token": lp.next_tok}
    for k, ref in pairs.items():
        assert torch.equal(out[k].view(torch.int32), ref.view(torch.int32)), k


def _forced_decisions(cm, mode_forced, fn):
    cm.cmsd_set_pass_decisions(mode_forced)
    try:
        out = fn()
        torch.cuda.synchronize()
        return {k: v.clone() for k, v in out.items() if isinstance(v, torch.Tensor)}
    finally:
        cm.cmsd_set_pass_decisions(0)


@pytest.mark.parametrize("adaptive", [False, True])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
def test_decision_paths_bitwise_equal(cm, name, mode, adaptive):
    # the decisions formed in every final-token workgroup (three launches) and read from
    # the decision kernel's record (four launches) are the same arithmetic: bit-equal
    # outputs; c2 and c3 choose the first by default, c4 the second
    cfg = W.CONFIGS[name]
    d = Hn.workload(name)
    run = lambda: _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max,
                        mode, adaptive)[0]
    rec = _forced_decisions(cm, 1, run)
    inl = _forced_decisions(cm, 2, run)
    auto = run()
    torch.cuda.synchronize()
    for k in ("draft_stats", "draft_len", "target_stats", "n_accepted", "next_token"):
        assert torch.equal(rec[k].view(torch.int32), inl[k].view(torch.int32)), k
        assert torch.equal(rec[k].view(torch.int32), auto[k].view(torch.int32)), k


@pytest.mark.parametrize("forced", [1, 2])
def test_decision_paths_invalid_sequence(cm, forced):
    V, K, B = 500, 4, 3
    g = np.random.default_rng(8)
    zd, zt, dr, u = _case(g, B, K, V, "f32")
    dr[1, 3] = V
    dev = torch.device("cuda:0")
    out = _forced_decisions(cm, forced, lambda: _pass(
        cm, Hn.to_device(zd, "f32", dev), Hn.to_device(zt, "f32", dev), torch.from_numpy(dr.reshape(-1)).to(dev),
        torch.from_numpy(u.reshape(-1)).to(dev), B, K, O.MODE_CM)[0])
    n_acc = out["n_accepted"].cpu().numpy()
    nxt = out["next_token"].cpu().numpy()
    ts = Hn.tstats_np(out["target_stats"])
    assert n_acc[1] == -1 and nxt[1] == -1 and ts["acc"][1 * (K + 1) + 3] == -2
    assert n_acc[0] >= 0 and n_acc[2] >= 0 and nxt[0] >= 0 and nxt[2] >= 0


def test_repeat_bitwise_identical(cm):
    cfg = W.CONFIGS["c2"]
    d = Hn.workload("c2")
    o1, _ = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, O.MODE_CM)
    o1 = {k: v.clone() for k, v in o1.items()}
    o2, _ = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, O.MODE_CM)
    for k in o1:
        assert torch.equal(o1[k].view(torch.int32), o2[k].view(torch.int32)), k


# ----------------------------------------------------------------------------- edge cases
def _case(g, B, K, V, dtype, scale=2.0, mask=None, mask_frac=0.0):
    # mask: columns masked (-inf) in every row; mask_frac: each row masks that share of
    # its logits at random, keeping at least one finite
    zd = g.normal(0, scale, (B * K, V)).astype(np.float32)
    zt = g.normal(0, scale, (B * (K + 1), V)).astype(np.float32)
    for b in range(B):
        for i in range(K):
            zt[b * (K + 1) + i] = zd[b * K + i] + g.normal(0, 0.5, V).astype(np.float32)
    if mask is not None:
        zd[:, mask] = -np.inf
        zt[:, mask] = -np.inf
    if mask_frac > 0.0:
        for z in (zd, zt):
            m = g.random(z.shape) < mask_frac
            m[np.arange(z.shape[0]), g.integers(0, V, z.shape[0])] = False
            z[m] = -np.inf
    store = (lambda x: x) if dtype == "f32" else W.bf16_bits_from_f32
    zds, zts = store(zd), store(zt)
    drafted = np.array([[int(np.argmax(Hn.decode(zds[b * K + i], dtype) + g.gumbel(size=V))) for i in range(K)]
                        for b in range(B)], dtype=np.int32)
    unif = (g.integers(0, 1 << 24, (B, K + 1)) * 2.0 ** -24).astype(np.float32)
    return zds, zts, drafted, unif


def _run_case(cm, zd, zt, drafted, unif, B, K, V, dtype, mode=O.MODE_CM, adaptive=False, pad=0, **kw):
    dev = torch.device("cuda:0")
    dd = Hn.to_device(zd, dtype, dev)
    td = Hn.to_device(zt, dtype, dev)
    if pad:
        # rows with a stride beyond the vocabulary
        dd = torch.nn.functional.pad(dd, (0, pad))[:, :V]
        td = torch.nn.functional.pad(td, (0, pad))[:, :V]
    out, P = _pass(cm, dd, td, torch.from_numpy(drafted.reshape(-1)).to(dev),
                   torch.from_numpy(unif.reshape(-1)).to(dev), B, K, mode, adaptive, **kw)
    t = Hn.Tally()
    n_acc, k = _check(t, B, K, V, dtype, zd, zt, drafted, unif, out, P, mode, adaptive, list(range(B)))
    t.assert_ok()
    return out, n_acc, k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V,K,B,pad", [(2, 1, 3, 0), (37, 3, 5, 3), (1000, 63, 2, 0), (4099, 5, 4, 5),
                                       (50257, 7, 3, 1), (300007, 2, 2, 0)])
def test_shapes(cm, dtype, V, K, B, pad):
    g = np.random.default_rng(V * 7 + K)
    zd, zt, dr, u = _case(g, B, K, V, dtype)
    for mode in (O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY):
        _run_case(cm, zd, zt, dr, u, B, K, V, dtype, mode=mode, adaptive=bool(mode == O.MODE_CM), pad=pad)


@pytest.mark.parametrize("seed", range(24))
def test_random_problems(cm, seed):
    # seeded random problems: vocabulary 2..70000 (log-uniform), 1..24 drafts, 1..6
    # sequences, either dtype, every mode, dense or adaptive lengths, padded strides,
    # per-row masks of random density or none, and each way the final-token workgroups
    # get their decisions; every output checked against the oracle
    g = np.random.default_rng(9000 + seed)
    V = int(round(math.exp(g.uniform(math.log(2), math.log(70000)))))
    K, B = int(g.integers(1, 25)), int(g.integers(1, 7))
    dtype = ("f32", "bf16")[int(g.integers(2))]
    mode = (O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY)[int(g.integers(3))]
    adaptive, pad = bool(g.integers(2)), int(g.integers(0, 6))
    mask_frac = (0.0, 0.0, 0.05, 0.5, 0.95)[int(g.integers(5))]
    decisions = int(g.integers(3))
    print(f"V={V} K={K} B={B} {dtype} mode={mode} adaptive={adaptive} pad={pad} mask={mask_frac} "
          f"decisions={decisions}", flush=True)
    zd, zt, dr, u = _case(g, B, K, V, dtype, scale=float(g.uniform(0.5, 4.0)), mask_frac=mask_frac)
    cm.cmsd_set_pass_decisions(decisions)
    try:
        _run_case(cm, zd, zt, dr, u, B, K, V, dtype, mode=mode, adaptive=adaptive, pad=pad)
    finally:
        cm.cmsd_set_pass_decisions(0)


@pytest.mark.parametrize("depth", [2, 3])
@pytest.mark.parametrize("block", [64, 128, 256])
def test_rounds_across_the_ring(cm, row_shape, block, depth):
    # drafter and target rows of 1..9 full 32-element-per-thread rounds (plus a partial
    # round and a tail), unaligned starts: every way through the streaming ring's main
    # loop and its last rounds, for every workgroup size and ring depth
    row_shape(block, depth)
    for nr in (1, 2, 3, 4, 5, 6, 9):
        V = 32 * block * nr + 37
        g = np.random.default_rng(nr * 100 + block)
        zd, zt, dr, u = _case(g, 2, 3, V, "bf16")
        _run_case(cm, zd, zt, dr, u, 2, 3, V, "bf16", mode=O.MODE_CM, adaptive=True, pad=1)


def test_masked_logits(cm):
    # -inf entries: flags bit 0, entropy over the finite entries, final tokens never masked
    V, K, B = 3001, 4, 4
    g = np.random.default_rng(5)
    mask = g.random(V) < 0.4
    zd, zt, dr, u = _case(g, B, K, V, "bf16", mask=mask)
    out, n_acc, _ = _run_case(cm, zd, zt, dr, u, B, K, V, "bf16")
    assert np.all(Hn.stats_np(out["draft_stats"])["flags"] & 1)
    assert not np.any(mask[out["next_token"].cpu().numpy()])


def test_invalid_drafted_id(cm):
    V, K, B = 500, 4, 3
    g = np.random.default_rng(8)
    zd, zt, dr, u = _case(g, B, K, V, "f32")
    dr[1, 3] = V          # out of range: sequence 1 is invalid, the others are not
    dev = torch.device("cuda:0")
    out, _ = _pass(cm, Hn.to_device(zd, "f32", dev), Hn.to_device(zt, "f32", dev),
                   torch.from_numpy(dr.reshape(-1)).to(dev), torch.from_numpy(u.reshape(-1)).to(dev), B, K,
                   O.MODE_CM)
    n_acc = out["n_accepted"].cpu().numpy()
    nxt = out["next_token"].cpu().numpy()
    ts = Hn.tstats_np(out["target_stats"])
    assert n_acc[1] == -1 and nxt[1] == -1 and ts["acc"][1 * (K + 1) + 3] == -2
    assert n_acc[0] >= 0 and n_acc[2] >= 0 and nxt[0] >= 0 and nxt[2] >= 0


def test_greedy_exact_match(cm):
    # top_beta = 0: exact-match verification; drafts equal to the target's top token
    # up to a chosen position are accepted, and the final token is that row's top token
    V, K, B = 2000, 6, 4
    g = np.random.default_rng(13)
    zd, zt, _, u = _case(g, B, K, V, "f32")
    dr = np.zeros((B, K), dtype=np.int32)
    for b in range(B):
        for i in range(K):
            top = int(np.argmax(zt[b * (K + 1) + i]))
            dr[b, i] = top if i < b + 1 else (top + 1) % V
    out, n_acc, _ = _run_case(cm, zd, zt, dr, u, B, K, V, "f32", mode=O.MODE_GREEDY, top_beta=0)
    nxt = out["next_token"].cpu().numpy()
    for b in range(B):
        assert n_acc[b] == b + 1
        assert nxt[b] == int(np.argmax(zt[b * (K + 1) + b + 1]))


def test_adaptive_lengths_cover_range(cm):
    # alpha sweeps k_b over [k_min, k_max]; the prefix never passes k_b and row k_b is final
    V, K, B = 4096, 8, 16
    g = np.random.default_rng(21)
    spikes = [(r, int(g.integers(0, V)), float(g.uniform(9, 22))) for r in range(B * K // 2)]
    zd, zt, dr, u = _case(g, B, K, V, "f32", scale=2.0)
    for r, v, h in spikes:       # the first half of the sequences: confident drafter rows
        zd[r, v] += h
        zt[(r // K) * (K + 1) + r % K, v] += h
        dr[r // K, r % K] = v
    seen = set()
    for alpha in (0.05, 0.3, 0.6, 1.0):
        out, n_acc, k = _run_case(cm, zd, zt, dr, u, B, K, V, "f32", adaptive=True, alpha=alpha)
        ts = Hn.tstats_np(out["target_stats"])
        assert np.all(n_acc <= k)
        assert all(ts["acc"][b * (K + 1) + k[b]] == -1 for b in range(B))
        seen |= set(k.tolist())
    assert min(seen) == 1 and max(seen) >= 6, seen


def test_empty_batch(cm):
    dev = torch.device("cuda:0")
    z = torch.zeros((0, 100), dtype=torch.float32, device=dev)
    out = cm.cmsd_logit_pass(z, z, torch.zeros(0, dtype=torch.int32, device=dev),
                             torch.zeros(0, dtype=torch.float32, device=dev), batch=0, k_max=4)
    torch.cuda.synchronize()
    assert out["n_accepted"].numel() == 0


def test_row_events_time_the_row_pass(cm):
    # events handed to the call are recorded around the row-pass launch on the call's
    # stream, and leave the outputs unchanged
    cfg = W.CONFIGS["c2"]
    d = Hn.workload("c2")
    ref, _ = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, O.MODE_CM)
    ref = {k: v.clone() for k, v in ref.items()}
    st = torch.cuda.Stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for e in ev:
        e.record(st)
    with pytest.raises(ValueError):
        cm.cmsd_logit_pass(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], batch=cfg.B,
                           k_max=cfg.k_max, row_events=ev[:1], stream=st)
    out = cm.cmsd_logit_pass(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], batch=cfg.B,
                             k_max=cfg.k_max, lambdas=Hn.PARAMS["lambdas"], beta_margin=Hn.PARAMS["beta_margin"],
                             k_min=Hn.PARAMS["k_min"], alpha=Hn.PARAMS["alpha"], mode=O.MODE_CM,
                             top_beta=Hn.PARAMS["top_beta"], tau_base=Hn.PARAMS["tau_base"],
                             gamma=Hn.PARAMS["gamma"], row_events=ev, stream=st)
    st.synchronize()
    ms = ev[0].elapsed_time(ev[1])
    assert 0.0 < ms < 100.0, ms
    for k in ref:
        assert torch.equal(out[k].view(torch.int32), ref[k].view(torch.int32)), k


def test_row_events_hook_is_one_shot(cm):
    # cmsd_set_row_events arms the next cmsd_logit_pass call only: a call the library
    # rejects disarms it, a later call records nothing, cmsd_logit_pass_noalloc neither
    # records nor disarms, and an armed call records around its row pass (1088 rows of
    # 50257 logits: tens of microseconds); unrecorded events keep their timestamps
    cfg = W.CONFIGS["c3"]
    d = Hn.workload("c3")
    st = torch.cuda.Stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for e in ev:
        e.record(st)
    st.synchronize()
    t0 = ev[0].elapsed_time(ev[1])

    def run(fn=cm.cmsd_logit_pass, **kw):
        fn(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], batch=cfg.B, k_max=cfg.k_max,
           stream=st, **kw)
        st.synchronize()

    cm.cmsd_set_row_events(ev)
    with pytest.raises(cm.CmsdError):
        run(top_beta=-1)                    # rejected on the host: the hook is disarmed
    run()
    assert ev[0].elapsed_time(ev[1]) == t0
    cm.cmsd_set_row_events(ev)
    run(fn=cm.cmsd_logit_pass_noalloc)      # not this call's hook
    assert ev[0].elapsed_time(ev[1]) == t0
    run()                                   # the armed call
    t1 = ev[0].elapsed_time(ev[1])
    assert t1 != t0 and 0.005 < t1 < 100.0, (t0, t1)
    run()
    assert ev[0].elapsed_time(ev[1]) == t1


class _DeviceRows:
    """Rows of a device bf16 matrix, fetched one at a time as stored bits."""

    def __init__(self, t):
        self.t = t

    def __getitem__(self, r):
        return self.t[r].view(torch.int16).cpu().numpy().view(np.uint16)


def test_large_batch_past_int32_elements(cm):
    # 1000 sequences of 16 drafts at V = 128256: 16000 drafter rows (2.05e9 logits) and
    # 17000 target rows (2.18e9), so element offsets pass 2^31 in both arrays; the
    # inputs come from torch's seeded generator on the device; sampled sequences at
    # the start, middle and end are checked against the oracle, and the three
    # separate calls must give the same bits
    from paper_2508_15371_amd import pipeline
    B, K, V = 1000, 16, 128256
    dev = torch.device("cuda:0")
    print(f"[logit pass large] B={B} K={K} V={V}", flush=True)
    g = torch.Generator(device=dev).manual_seed(1234)
    sig = torch.exp(torch.empty(B * K, 1, device=dev).uniform_(math.log(0.3), math.log(10.0), generator=g))
    draft = torch.empty(B * K, V, dtype=torch.bfloat16, device=dev)
    target = torch.empty(B * (K + 1), V, dtype=torch.bfloat16, device=dev)
    drafted = torch.empty(B * K, dtype=torch.int32, device=dev)
    for c0 in range(0, B, 100):               # 100 sequences at a time
        c1 = c0 + 100
        z = torch.randn((c1 - c0) * K, V, device=dev, generator=g) * sig[c0 * K:c1 * K]
        draft[c0 * K:c1 * K] = z.to(torch.bfloat16)
        zd = draft[c0 * K:c1 * K].float()
        gum = -torch.log(-torch.log(torch.rand(zd.shape, device=dev, generator=g).clamp_(1e-12, 1.0 - 1e-7)))
        drafted[c0 * K:c1 * K] = torch.argmax(zd + gum, dim=1).to(torch.int32)
        t3 = target[c0 * (K + 1):c1 * (K + 1)].view(c1 - c0, K + 1, V)
        t3[:, :K] = (zd + 0.5 * torch.randn(zd.shape, device=dev, generator=g)).view(c1 - c0, K, V).to(torch.bfloat16)
        t3[:, K] = (2.0 * torch.randn(c1 - c0, V, device=dev, generator=g)).to(torch.bfloat16)
        del z, zd, gum
    unif = (torch.randint(0, 1 << 24, (B * (K + 1),), device=dev, generator=g).float() * 2.0 ** -24).contiguous()
    out, P = _pass(cm, draft, target, drafted, unif, B, K, O.MODE_CM)
    t = Hn.Tally()
    n_acc, _ = _check(t, B, K, V, "bf16", _DeviceRows(draft), _DeviceRows(target), drafted.view(B, K).cpu().numpy(),
                      unif.view(B, K + 1).cpu().numpy(), out, P, O.MODE_CM, False, [0, 1, 499, 998, 999])
    print(f"[logit pass large] checked={t.checked} exceptions={t.exceptions} mean n_acc={n_acc.mean():.3f}", flush=True)
    t.assert_ok()
    lp = pipeline.LogitPass(B, K, V, dev, pipeline.Params(mode=O.MODE_CM))
    lp.run(draft, target, drafted, unif)
    torch.cuda.synchronize()
    for k, ref in {"draft_stats": lp.stats, "draft_len": lp.k, "target_stats": lp.tstats, "n_accepted": lp.n_acc,
                   "next_token": lp.next_tok}.items():
        assert torch.equal(out[k].view(torch.int32), ref.view(torch.int32)), k


@pytest.mark.parametrize("mode", [O.MODE_CM, O.MODE_GREEDY])
def test_graph_capture_replays_match_eager(cm, mode):
    # one cmsd_logit_pass call allocates and synchronises nothing, so it can be captured
    # in a HIP graph: every replay (with eager work in between) matches the eager run
    from paper_2508_15371_amd import pipeline
    cfg = W.CONFIGS["c3"]
    d = Hn.workload("c3")
    args = (d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"])
    ref = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", pipeline.Params(mode=mode))
    ref.logit_pass(*args)
    torch.cuda.synchronize()
    fields = ("stats", "k", "tstats", "n_acc", "next_tok")
    want = {f: getattr(ref, f).clone() for f in fields}
    lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", pipeline.Params(mode=mode))
    lp.logit_pass(*args)                           # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lp.logit_pass(*args)
    junk = torch.zeros(1 << 20, device="cuda:0")
    for rep in range(4):
        lp.stats.fill_(float("nan"))
        lp.tstats.fill_(float("nan"))
        lp.k.fill_(-7)
        lp.n_acc.fill_(-7)
        lp.next_tok.fill_(-7)
        junk.add_(1.0)                             # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for f in fields:
            a, b = getattr(lp, f), want[f]
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (rep, f)


@pytest.mark.parametrize("mode,kw", [
    (O.MODE_CM, dict(gamma=-1.0)),                               # the prose's direction: confident -> lenient
    (O.MODE_CM, dict(gamma=3.0, tau_base=0.0)),
    (O.MODE_CM, dict(top_beta=1, tau_base=2.0, gamma=0.0)),
    (O.MODE_CM, dict(top_beta=10, tau_base=0.5)),
    (O.MODE_CM, dict(top_beta=0)),                               # gate off: standard speculative sampling
    (O.MODE_CM, dict(alpha=0.3, k_min=2)),
    (O.MODE_CM, dict(lambdas=(1.0, 0.0, 0.0), beta_margin=0.25)),
    (O.MODE_GREEDY, dict(top_beta=1, tau_base=0.0, gamma=-0.5)),
    (O.MODE_GREEDY, dict(top_beta=5, tau_base=1.0, gamma=2.0)),
], ids=["gamma-1", "gamma3-tau0", "beta1-tau2", "beta10", "beta0", "alpha0.3-kmin2", "entropy-only",
        "greedy-beta1", "greedy-beta5"])
@pytest.mark.parametrize("adaptive", [False, True])
def test_parameter_settings(cm, mode, kw, adaptive):
    # the gate, threshold, draft-length and confidence parameters away from their
    # defaults, on c3 (odd V), 16 sequences against the oracle
    cfg = W.CONFIGS["c3"]
    d = Hn.workload("c3")
    out, P = _pass(cm, d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], cfg.B, cfg.k_max, mode,
                   adaptive, **kw)
    t = Hn.Tally()
    n_acc, k = _check(t, cfg.B, cfg.k_max, cfg.V, cfg.dtype, d["draft"], d["target"], d["drafted"], d["uniforms"],
                      out, P, mode, adaptive, _seqs(cfg.B, 16, 77), stats_rows=False)
    print(f"[logit pass params] {kw} mode={mode} adaptive={adaptive}: checked={t.checked} exceptions={t.exceptions} "
          f"mean n_acc={n_acc.mean():.3f} mean k={k.mean():.3f}", flush=True)
    t.assert_ok()


def test_boundary_uniforms(cm):
    # u = 0 and u = 1 - 2^-24, the ends of the uniform grid, with outcomes fixed by
    # construction: target rows 0..K-1 equal the drafter rows except tokens j < k
    # raised by 2 and 1, so p_t > p_d exactly there (the residual lives on {j, k}) and
    # p_t < p_d elsewhere; the final rows mask everything outside [lo, hi]
    B, K, V = 4, 2, 4099
    g = np.random.default_rng(2024)
    zd = g.normal(0, 1, (B * K, V)).astype(np.float32)
    zt = np.zeros((B * (K + 1), V), dtype=np.float32)
    boost = {}
    for b in range(B):
        for i in range(K):
            j, k = sorted(g.choice(V, 2, replace=False).tolist())
            boost[(b, i)] = (j, k)
            row = zd[b * K + i].copy()
            row[j] += 2.0
            row[k] += 1.0
            zt[b * (K + 1) + i] = row
        fin = np.full(V, -np.inf, dtype=np.float32)
        lo, hi = 100 + b, V - 50 - b
        fin[lo:hi + 1] = g.normal(0, 1, hi - lo + 1).astype(np.float32)
        fin[hi] = 3.0                                       # a large final mass at the last live token
        zt[b * (K + 1) + K] = fin
        boost[(b, "final")] = (lo, hi)
    top = 1.0 - 2.0 ** -24
    # sequence 0: boosted drafts (ratio > 1) pass even at u = 1 - 2^-24; bonus with u = 0
    # sequence 1: an unboosted draft (ratio < 1) fails at u = 1 - 2^-24; residual with u = 0
    # sequence 2: the same rejection; residual with u = 1 - 2^-24
    # sequence 3: drafts accepted at u = 0 (p_t > 0); bonus with u = 1 - 2^-24
    dr = np.zeros((B, K), dtype=np.int32)
    un = np.zeros((B, K + 1), dtype=np.float32)
    dr[0] = [boost[(0, 0)][0], boost[(0, 1)][1]]
    un[0] = [top, top, 0.0]
    for b in (1, 2):
        j, k = boost[(b, 0)]
        dr[b] = [(j + k) // 2 if (j + k) // 2 not in (j, k) else (k + 1) % V, 0]
        un[b] = [top, 0.5, 0.0 if b == 1 else top]
    dr[3] = [7, 11]
    un[3] = [0.0, 0.0, top]
    dev = torch.device("cuda:0")
    out, P = _pass(cm, Hn.to_device(zd, "f32", dev), Hn.to_device(zt, "f32", dev), torch.from_numpy(dr.reshape(-1)).to(dev),
                   torch.from_numpy(un.reshape(-1)).to(dev), B, K, O.MODE_STANDARD)
    n_acc = out["n_accepted"].cpu().tolist()
    nxt = out["next_token"].cpu().tolist()
    assert n_acc == [2, 0, 0, 2], n_acc
    assert nxt[0] == boost[(0, "final")][0]                 # u = 0: the first live token of the bonus row
    assert nxt[1] == boost[(1, 0)][0]                        # u = 0: the first residual token j
    assert nxt[2] == boost[(2, 0)][1]                        # u = 1 - 2^-24: the last residual token k
    assert nxt[3] == boost[(3, "final")][1]                 # u = 1 - 2^-24: the last live token (large mass)
    # and the oracle agrees on every one
    for b in range(B):
        res = O.verify_sequence([zt[b * (K + 1) + i].astype(np.float64) for i in range(K + 1)],
                                [zd[b * K + i].astype(np.float64) for i in range(K)], dr[b],
                                [float(u) for u in un[b]], [0.5] * K, K, O.MODE_STANDARD, 3, 0.1, 1.0)
        assert (res["n_acc"], res["next"]) == (n_acc[b], nxt[b]), b
