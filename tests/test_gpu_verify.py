"""GPU parity of cmsd_draft_len (Sec. III.B(b)) and cmsd_verify (Sec. III.A, III.B(c))
against the oracle, through the C ABI, on the five workloads and edge cases."""
import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import cmsd_oracle as O
from tests import harness as Hn

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mods():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_15371_amd import cmsd, pipeline
    return cmsd, pipeline


def _params(pipeline, mode):
    P = Hn.PARAMS
    return pipeline.Params(lambdas=P["lambdas"], beta_margin=P["beta_margin"], k_min=P["k_min"], alpha=P["alpha"],
                           mode=mode, top_beta=P["top_beta"], tau_base=P["tau_base"], gamma=P["gamma"])


def _run(mods, name, mode, seed=0):
    cmsd, pipeline = mods
    cfg = W.CONFIGS[name]
    d = Hn.workload(name, seed)
    lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", _params(pipeline, mode), dense=not cfg.ragged)
    lp.confidence(d["draft_dev"])
    lp.draft_len()
    if cfg.ragged:
        target = W.pack_device(d["target_dev"], lp.k, lp.off, cfg.k_max)
        unif = W.pack_device(d["unif_dev"], lp.k, lp.off, cfg.k_max)
    else:
        target, unif = d["target_dev"], d["unif_dev"]
    lp.verify(d["draft_dev"], target, d["drafted_dev"], unif)
    torch.cuda.synchronize()
    return cfg, d, lp


def _sample_seqs(cfg, n):
    if cfg.B <= n:
        return list(range(cfg.B))
    g = np.random.default_rng(100 + cfg.cid)
    return sorted(set([0, cfg.B - 1] + g.choice(cfg.B, n, replace=False).tolist()))


def _check_draft_len(t, cfg, d, gs, k_gpu, off_gpu, seqs):
    K = cfg.k_max
    P = Hn.PARAMS
    # stage isolation: the oracle's draft length on the GPU's confidences is bit-exact
    Cg = gs["C"].astype(np.float64).reshape(cfg.B, K)
    k_o, off_o, _ = O.draft_len(Cg, P["k_min"], K, Hn.f32(P["alpha"]))
    t.value("k(stage)", np.array_equal(k_o, k_gpu), (k_o[:8], k_gpu[:8]))
    t.value("off(stage)", np.array_equal(off_o, off_gpu), (off_o[:8], off_gpu[:8]))
    # end to end on sampled sequences: the oracle's own confidences
    for b in seqs:
        C = np.array([[Hn.oracle_conf(Hn.decode(d["draft"][b * K + i], cfg.dtype), cfg.V) for i in range(K)]])
        kb, _, sl = O.draft_len(C, P["k_min"], K, Hn.f32(P["alpha"]))
        t.decision(f"k[{b}]", int(k_gpu[b]), int(kb[0]), float(sl[0]))


def _verify_check(mods, name, mode, nseq):
    cfg, d, lp = _run(mods, name, mode)
    K, V = cfg.k_max, cfg.V
    gs = Hn.stats_np(lp.stats)
    ts = Hn.tstats_np(lp.tstats)
    k_gpu = lp.k.cpu().numpy()
    off_gpu = lp.off.cpu().numpy()
    n_acc = lp.n_acc.cpu().numpy()
    nxt = lp.next_tok.cpu().numpy()
    t = Hn.Tally()
    seqs = _sample_seqs(cfg, nseq)
    _check_draft_len(t, cfg, d, gs, k_gpu, off_gpu, seqs[: max(4, len(seqs) // 2)])
    for b in seqs:
        kb = int(k_gpu[b]) if cfg.ragged else K
        toff = int(off_gpu[b]) if cfg.ragged else b * (K + 1)
        zd = [Hn.decode(d["draft"][b * K + i], cfg.dtype) for i in range(K)]
        pos = list(range(kb)) + [K]
        zt = [Hn.decode(d["target"][b * (K + 1) + i], cfg.dtype) for i in pos]
        unif = [float(d["uniforms"][b, i]) for i in pos]
        C = [Hn.oracle_conf(z, V) for z in zd]
        Hn.check_sequence(t, b, zt, zd, d["drafted"][b], unif, C, kb, mode, Hn.PARAMS, ts, toff,
                          int(n_acc[b]), int(nxt[b]))
    print(f"[verify parity] {name} mode={mode}: checked={t.checked} exceptions={t.exceptions} "
          f"mean n_acc={n_acc.mean():.3f} mean k={k_gpu.mean():.3f}", flush=True)
    t.assert_ok()
    return t


@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
@pytest.mark.parametrize("name,nseq", [("tiny", 1), ("c2", 8), ("c3", 64), ("c4", 6), ("c5", 24), ("v152k", 8)])
def test_verify_configs(mods, name, nseq, mode):
    print(f"[verify parity] start {name} mode={mode}", flush=True)
    _verify_check(mods, name, mode, nseq)


def test_verify_repeat_bitwise_identical(mods):
    cfg, d, lp = _run(mods, "c3", O.MODE_CM)
    a = (lp.n_acc.clone(), lp.next_tok.clone(), lp.tstats.clone())
    cfg, d, lp2 = _run(mods, "c3", O.MODE_CM)
    assert torch.equal(a[0], lp2.n_acc) and torch.equal(a[1], lp2.next_tok)
    assert torch.equal(a[2].view(torch.int32), lp2.tstats.view(torch.int32))


# ----------------------------------------------------------------------------- edge cases
def _small_case(g, B, K, V, dtype, scale=2.0, mask_frac=0.0):
    # mask_frac: each row masks (-inf) that share of its logits at random, keeping one finite
    zd = (g.normal(0, scale, (B * K, V))).astype(np.float32)
    zt = (g.normal(0, scale, (B * (K + 1), V))).astype(np.float32)
    for b in range(B):
        for i in range(K):
            zt[b * (K + 1) + i] = zd[b * K + i] + g.normal(0, 0.5, V).astype(np.float32)
    if mask_frac > 0.0:
        for z in (zd, zt):
            m = g.random(z.shape) < mask_frac
            m[np.arange(z.shape[0]), g.integers(0, V, z.shape[0])] = False
            z[m] = -np.inf
    store = (lambda x: x) if dtype == "f32" else W.bf16_bits_from_f32
    drafted = np.array([[int(np.argmax(Hn.decode(store(zd[b * K + i]), dtype) + g.gumbel(size=V)))
                         for i in range(K)] for b in range(B)], dtype=np.int32)
    unif = (g.integers(0, 1 << 24, (B, K + 1)) * 2.0 ** -24).astype(np.float32)
    return store(zd), store(zt), drafted, unif


def _run_small(mods, zd, zt, drafted, unif, k, dtype, B, K, V, mode=O.MODE_CM, top_beta=3, tau_base=0.1,
               gamma=1.0, off=None):
    cmsd, _ = mods
    dev = torch.device("cuda:0")
    dd = Hn.to_device(zd, dtype, dev)
    td = Hn.to_device(zt, dtype, dev)
    st = cmsd.cmsd_confidence(dd)
    if off is None:
        off = np.concatenate([[0], np.cumsum(np.asarray(k) + 1)]).astype(np.int32)
    n_acc, nxt, ts = cmsd.cmsd_verify(
        dd, st, td, torch.from_numpy(off).to(dev), torch.from_numpy(np.asarray(k, dtype=np.int32)).to(dev),
        torch.from_numpy(drafted.reshape(-1)).to(dev), torch.from_numpy(unif.reshape(-1)).to(dev),
        batch=B, k_max=K, mode=mode, top_beta=top_beta, tau_base=tau_base, gamma=gamma)
    torch.cuda.synchronize()
    return Hn.stats_np(st), n_acc.cpu().numpy(), nxt.cpu().numpy(), Hn.tstats_np(ts)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V", [2, 5, 64, 1000, 4097, 32003])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
def test_ragged_lengths_small_vocab(mods, dtype, V, mode):
    # packed target rows with every draft length 0..K (k_b = 0: bonus sample only)
    g = np.random.default_rng(V + 31 * mode)
    B, K = 6, 5
    zd, zt_pad, drafted, unif_pad = _small_case(g, B, K, V, dtype)
    k = np.array([0, 1, 5, 3, 2, 4], dtype=np.int32)
    zt = W.pack_ragged(k, K, zt_pad.reshape(B, K + 1, V))
    unif = W.pack_ragged(k, K, unif_pad.reshape(B, K + 1, 1)).reshape(-1)
    off = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    gs, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, dtype, B, K, V, mode=mode)
    t = Hn.Tally()
    for b in range(B):
        kb = int(k[b])
        zdr = [Hn.decode(zd[b * K + i], dtype) for i in range(K)]
        ztr = [Hn.decode(zt[off[b] + i], dtype) for i in range(kb + 1)]
        C = [Hn.oracle_conf(z, V) for z in zdr]
        Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[off[b]:off[b] + kb + 1], C, kb, mode, Hn.PARAMS,
                          ts, int(off[b]), int(n_acc[b]), int(nxt[b]))
    t.assert_ok()


@pytest.mark.parametrize("seed", range(16))
def test_random_ragged_problems(mods, seed):
    # seeded random ragged problems through cmsd_confidence + cmsd_verify: vocabulary
    # 2..70000 (log-uniform), up to 16 drafts (every fourth case up to 80, past one
    # wave's 64 positions), 1..8 sequences with draft lengths drawn from 0..k_max and
    # their target rows packed, either dtype, every mode, random gate parameters, per-row
    # masks of random density or none; every output against the oracle
    g = np.random.default_rng(7000 + seed)
    V = int(round(math.exp(g.uniform(math.log(2), math.log(70000)))))
    K = int(g.integers(1, 81 if seed % 4 == 3 else 17))
    B = int(g.integers(1, 9))
    dtype = ("f32", "bf16")[int(g.integers(2))]
    mode = (O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY)[int(g.integers(3))]
    mask_frac = (0.0, 0.0, 0.05, 0.5, 0.95)[int(g.integers(5))]
    top_beta = int(g.choice([0, 1, 3, 10]))
    tau_base, gamma = float(g.uniform(0.0, 1.0)), float(g.uniform(-1.0, 2.0))
    print(f"V={V} K={K} B={B} {dtype} mode={mode} mask={mask_frac} beta={top_beta} tau={tau_base:.3f} "
          f"gamma={gamma:.3f}", flush=True)
    zd, zt_pad, drafted, unif_pad = _small_case(g, B, K, V, dtype, scale=float(g.uniform(0.5, 4.0)),
                                                mask_frac=mask_frac)
    k = g.integers(0, K + 1, B).astype(np.int32)
    zt = W.pack_ragged(k, K, zt_pad.reshape(B, K + 1, V))
    unif = W.pack_ragged(k, K, unif_pad.reshape(B, K + 1, 1)).reshape(-1)
    off = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    gs, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, dtype, B, K, V, mode=mode, top_beta=top_beta,
                                    tau_base=tau_base, gamma=gamma)
    P = dict(Hn.PARAMS, top_beta=top_beta, tau_base=tau_base, gamma=gamma)
    t = Hn.Tally()
    for b in range(B):
        kb = int(k[b])
        zdr = [Hn.decode(zd[b * K + i], dtype) for i in range(K)]
        for i in range(K):
            Hn.check_row_stats(t, gs, b * K + i, zdr[i], V, tuple(Hn.f32(x) for x in P["lambdas"]),
                               Hn.f32(P["beta_margin"]))
        ztr = [Hn.decode(zt[off[b] + i], dtype) for i in range(kb + 1)]
        C = [Hn.oracle_conf(z, V) for z in zdr]
        Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[off[b]:off[b] + kb + 1], C, kb, mode, P,
                          ts, int(off[b]), int(n_acc[b]), int(nxt[b]))
    t.assert_ok()


@pytest.mark.parametrize("block", [64, 128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
def test_each_row_block(mods, row_shape, block, dtype, mode):
    # every workgroup size the library may pick for the target-row pass
    row_shape(block)
    g = np.random.default_rng(block + 7 * mode)
    B, K, V = 5, 4, 9001
    zd, zt_pad, drafted, unif_pad = _small_case(g, B, K, V, dtype)
    k = np.array([4, 0, 2, 3, 1], dtype=np.int32)
    zt = W.pack_ragged(k, K, zt_pad.reshape(B, K + 1, V))
    unif = W.pack_ragged(k, K, unif_pad.reshape(B, K + 1, 1)).reshape(-1)
    off = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    gs, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, dtype, B, K, V, mode=mode)
    t = Hn.Tally()
    for b in range(B):
        kb = int(k[b])
        zdr = [Hn.decode(zd[b * K + i], dtype) for i in range(K)]
        ztr = [Hn.decode(zt[off[b] + i], dtype) for i in range(kb + 1)]
        C = [Hn.oracle_conf(z, V) for z in zdr]
        Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[off[b]:off[b] + kb + 1], C, kb, mode, Hn.PARAMS,
                          ts, int(off[b]), int(n_acc[b]), int(nxt[b]))
    t.assert_ok()


@pytest.mark.parametrize("dtype,V", [("f32", 300007), ("bf16", 600011)])
@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
def test_vocab_beyond_one_slice_per_thread(mods, dtype, V, mode):
    # more than 256 vocabulary slices: the sampling pass runs several slices per thread
    g = np.random.default_rng(V + mode)
    B, K = 3, 2
    zd, zt_pad, drafted, unif_pad = _small_case(g, B, K, V, dtype)
    k = np.array([2, 0, 1], dtype=np.int32)
    zt = W.pack_ragged(k, K, zt_pad.reshape(B, K + 1, V))
    unif = W.pack_ragged(k, K, unif_pad.reshape(B, K + 1, 1)).reshape(-1)
    off = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    gs, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, dtype, B, K, V, mode=mode)
    t = Hn.Tally()
    for b in range(B):
        kb = int(k[b])
        zdr = [Hn.decode(zd[b * K + i], dtype) for i in range(K)]
        ztr = [Hn.decode(zt[off[b] + i], dtype) for i in range(kb + 1)]
        C = [Hn.oracle_conf(z, V) for z in zdr]
        Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[off[b]:off[b] + kb + 1], C, kb, mode, Hn.PARAMS,
                          ts, int(off[b]), int(n_acc[b]), int(nxt[b]))
    t.assert_ok()


def test_equal_rows_accept_everything_and_masked_targets(mods):
    g = np.random.default_rng(5)
    B, K, V = 4, 6, 3000
    zd, zt, drafted, unif = _small_case(g, B, K, V, "bf16")
    for b in range(B):
        for i in range(K):
            zt[b * (K + 1) + i] = zd[b * K + i]
    unif[:, :K] = np.float32(1.0 - 2.0 ** -24)
    k = np.full(B, K, dtype=np.int32)
    for mode in (O.MODE_STANDARD, O.MODE_CM):
        _, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, "bf16", B, K, V, mode=mode)
        assert (n_acc == K).all()
    # a drafted token with zero target mass is always rejected
    zt2 = zt.copy()
    ninf = W.bf16_bits_from_f32(np.array([-np.inf], dtype=np.float32))[0]
    for b in range(B):
        zt2[b * (K + 1) + 2, drafted[b, 2]] = ninf
    unif2 = np.zeros_like(unif)
    _, n_acc, nxt, ts = _run_small(mods, zd, zt2, drafted, unif2, k, "bf16", B, K, V, mode=O.MODE_CM,
                                   top_beta=V, tau_base=1e30, gamma=0.0)
    assert (n_acc == 2).all()
    for b in range(B):
        assert Hn.decode(zt2[b * (K + 1) + 2], "bf16")[nxt[b]] > -math.inf


def test_invalid_device_inputs_are_reported(mods):
    g = np.random.default_rng(6)
    B, K, V = 4, 3, 500
    zd, zt, drafted, unif = _small_case(g, B, K, V, "f32")
    k = np.full(B, K, dtype=np.int32)
    drafted_bad = drafted.copy()
    drafted_bad[1, 1] = V            # out of range id
    drafted_bad[2, 0] = -5
    _, n_acc, nxt, _ = _run_small(mods, zd, zt, drafted_bad, unif, k, "f32", B, K, V)
    assert n_acc[1] == -1 and nxt[1] == -1 and n_acc[2] == -1 and nxt[2] == -1
    assert n_acc[0] >= 0 and n_acc[3] >= 0
    k_bad = k.copy()
    k_bad[3] = K + 1                 # longer than k_max
    off = np.arange(B + 1, dtype=np.int32) * (K + 1)
    _, n_acc, nxt, _ = _run_small(mods, zd, zt, drafted, unif, k_bad, "f32", B, K, V, off=off)
    assert n_acc[3] == -1 and (n_acc[:3] >= 0).all()
    off_bad = off.copy()
    off_bad[B] = B * (K + 1) + 50    # beyond the allocated target rows
    _, n_acc, nxt, _ = _run_small(mods, zd, zt, drafted, unif, k, "f32", B, K, V, off=off_bad)
    assert n_acc[B - 1] == -1 and (n_acc[: B - 1] >= 0).all()


def test_draft_len_edges(mods):
    cmsd, _ = mods
    dev = torch.device("cuda:0")
    g = np.random.default_rng(8)
    # (1500, 40) and (5, 4096): sequences straddle the 16384-value staging chunks
    for B, K, kmin, alpha in ((0, 4, 1, 1.0), (1, 1, 1, 1.0), (3000, 16, 2, 0.61), (700, 7, 7, 0.3),
                              (1500, 40, 3, 0.9), (5, 4096, 1, 1.0)):
        C = g.uniform(0, 1, B * K).astype(np.float32)
        st = torch.zeros((B * K, 8), dtype=torch.float32)
        st[:, 5] = torch.from_numpy(C)
        k, off = cmsd.cmsd_draft_len(st.to(dev), B, k_min=kmin, k_max=K, alpha=alpha)
        torch.cuda.synchronize()
        k_o, off_o, _ = O.draft_len(C.astype(np.float64).reshape(B, K), kmin, K, Hn.f32(alpha))
        assert np.array_equal(k.cpu().numpy(), k_o)
        assert np.array_equal(off.cpu().numpy(), off_o)


def test_greedy_exact_match_on_device(mods):
    # top_beta = 0 (gate off): exact-match verification against the lowest index of
    # the target max; drafts hit it at a seeded subset of positions, and some rows get
    # a tied max at a higher index that the draft names (rejected); no uniforms
    cmsd, _ = mods
    g = np.random.default_rng(21)
    B, K, V = 16, 8, 5000
    zd, zt, drafted, _ = _small_case(g, B, K, V, "bf16")
    for b in range(B):
        for i in range(K):
            r = b * (K + 1) + i
            z = Hn.decode(zt[r], "bf16")
            top = int(np.argmax(z))
            u = g.random()
            if u < 0.7:
                drafted[b, i] = top
            elif u < 0.8 and top < V - 1:
                hi = int(g.integers(top + 1, V))
                zt[r, hi] = zt[r, top]          # tied max at a higher index
                drafted[b, i] = hi
    ztd = np.stack([Hn.decode(zt[r], "bf16") for r in range(B * (K + 1))])
    dev = torch.device("cuda:0")
    dd, td = Hn.to_device(zd, "bf16", dev), Hn.to_device(zt, "bf16", dev)
    st = cmsd.cmsd_confidence(dd)
    k = torch.full((B,), K, dtype=torch.int32, device=dev)
    off = (torch.arange(B + 1, dtype=torch.int32, device=dev) * (K + 1)).contiguous()
    n_acc, nxt, ts = cmsd.cmsd_verify(dd, st, td, off, k, torch.from_numpy(drafted.reshape(-1)).to(dev), None,
                                      batch=B, k_max=K, mode=cmsd.CMSD_MODE_GREEDY, top_beta=0, tau_base=0.5,
                                      gamma=1.0)
    torch.cuda.synchronize()
    n_acc, nxt = n_acc.cpu().numpy(), nxt.cpu().numpy()
    for b in range(B):
        c = 0
        while c < K and drafted[b, c] == int(np.argmax(ztd[b * (K + 1) + c])):
            c += 1
        assert n_acc[b] == c
        assert nxt[b] == int(np.argmax(ztd[b * (K + 1) + c]))


@pytest.mark.parametrize("mode", [O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY])
@pytest.mark.parametrize("K", [63, 64, 70, 130])
def test_long_drafts(mods, mode, K):
    # draft lengths around and beyond one wavefront of positions (the prefix scan and
    # the final pass read a sequence's positions 64 at a time)
    g = np.random.default_rng(K * 3 + mode)
    B, V = 4, 300
    zd, zt_pad, drafted, unif_pad = _small_case(g, B, K, V, "f32", scale=0.4)
    # targets equal to the drafts except a few positions, so prefixes run long
    for b in range(B):
        for i in range(K):
            zt_pad[b * (K + 1) + i] = zd[b * K + i]
    for b, i in ((0, 5), (1, 63), (1, K - 1), (2, min(64, K - 1))):
        zt_pad[b * (K + 1) + i] = g.normal(0, 3, V).astype(np.float32)
    unif_pad[:, :K] = np.float32(0.9)
    k = np.array([K, K, min(64, K), K - 1], dtype=np.int32)
    zt = W.pack_ragged(k, K, zt_pad.reshape(B, K + 1, V))
    unif = W.pack_ragged(k, K, unif_pad.reshape(B, K + 1, 1)).reshape(-1)
    off = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    prm = dict(Hn.PARAMS, top_beta=1, tau_base=0.0, gamma=0.0) if mode == O.MODE_GREEDY else Hn.PARAMS
    gs, n_acc, nxt, ts = _run_small(mods, zd, zt, drafted, unif, k, "f32", B, K, V, mode=mode,
                                    top_beta=prm["top_beta"], tau_base=prm["tau_base"], gamma=prm["gamma"])
    t = Hn.Tally()
    for b in range(B):
        kb = int(k[b])
        zdr = [Hn.decode(zd[b * K + i], "f32") for i in range(K)]
        ztr = [Hn.decode(zt[off[b] + i], "f32") for i in range(kb + 1)]
        C = [Hn.oracle_conf(z, V) for z in zdr]
        Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[off[b]:off[b] + kb + 1], C, kb, mode, prm, ts,
                          int(off[b]), int(n_acc[b]), int(nxt[b]))
    t.assert_ok()


def test_side_stream_matches_default_stream(mods):
    # every call enqueues on the stream it is given: a full iteration on a side
    # stream, ordered after the uploads by an event, gives the default stream's
    # results bit for bit
    cmsd, pipeline = mods
    cfg = W.CONFIGS["c2"]
    d = Hn.workload("c2", 0)
    outs = []
    for use_side in (False, True):
        lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", _params(pipeline, O.MODE_CM))
        if use_side:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                lp.run(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"], stream=side)
            torch.cuda.current_stream().wait_stream(side)
        else:
            lp.run(d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"])
        torch.cuda.synchronize()
        outs.append([x.cpu().clone() for x in (lp.stats, lp.k, lp.off, lp.tstats, lp.n_acc, lp.next_tok)])
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           b.view(torch.int32) if b.dtype == torch.float32 else b)


def test_graph_capture_replays_match_eager(mods):
    # the iteration allocates nothing and synchronises nothing, so it can be captured
    # in a HIP graph: every replay (with eager work in between) matches the eager run
    cmsd, pipeline = mods
    cfg = W.CONFIGS["c2"]
    d = Hn.workload("c2", 0)
    args = (d["draft_dev"], d["target_dev"], d["drafted_dev"], d["unif_dev"])
    ref = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", _params(pipeline, O.MODE_CM))
    ref.run(*args)
    torch.cuda.synchronize()
    want = [x.clone() for x in (ref.stats, ref.k, ref.off, ref.tstats, ref.n_acc, ref.next_tok)]
    lp = pipeline.LogitPass(cfg.B, cfg.k_max, cfg.V, "cuda:0", _params(pipeline, O.MODE_CM))
    lp.run(*args)                                  # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lp.run(*args)
    junk = torch.zeros(1 << 20, device="cuda:0")
    for rep in range(4):
        for x in (lp.stats, lp.tstats):
            x.fill_(float("nan"))
        lp.n_acc.fill_(-7)
        lp.next_tok.fill_(-7)
        junk.add_(1.0)                             # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (lp.stats, lp.k, lp.off, lp.tstats, lp.n_acc, lp.next_tok)
        for a, b in zip(got, want):
            assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                               b.view(torch.int32) if b.dtype == torch.float32 else b), rep


@pytest.mark.parametrize("conf_block", [64, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V", [4, 3001, 50257])
def test_zero_residual_falls_back_to_target_row(mods, row_shape, conf_block, dtype, V):
    # Drafter and target rows equal at every drafted position; sequence b's draft at
    # position c_b = b % K is a token both rows mask (-inf), rejected with certainty,
    # and the residual of two equal rows is identically zero: the final token is
    # sampled from p_t of row c_b (reading R13).  The earlier drafts are the rows' top
    # tokens (always accepted: p_t = p_d).  The drafter stats come from a launch of
    # another workgroup size than the target rows' (conf_block 64), so their
    # normalisers may differ in the last bits: the final-token pass then meets a slice
    # mass of rounding size whose exact weights are all zero, the second way to the
    # fallback; with equal sizes the slice masses are exactly zero.
    cmsd, _ = mods
    g = np.random.default_rng(V * 3 + conf_block + (dtype == "bf16"))
    B, K = 6, 4
    store = (lambda x: x.astype(np.float32)) if dtype == "f32" else W.bf16_bits_from_f32
    zd = store(g.normal(0, 2.0, (B * K, V)))
    drafted = np.zeros((B, K), dtype=np.int32)
    cs = []
    for b in range(B):
        c = b % (K + 1)            # c = K: nothing masked, every draft accepted, bonus row
        cs.append(c)
        for i in range(K):
            r = b * K + i
            z = Hn.decode(zd[r], dtype)
            if i == c:
                y = int(g.integers(0, V))
                while y == int(np.argmax(z)):
                    y = int(g.integers(0, V))
                zd[r, y] = 0xFF80 if dtype == "bf16" else -np.inf     # -inf in the stored dtype
                drafted[b, i] = y
            else:
                drafted[b, i] = int(np.argmax(z))
    zt = np.empty((B * (K + 1), V), dtype=zd.dtype)
    for b in range(B):
        zt[b * (K + 1):b * (K + 1) + K] = zd[b * K:(b + 1) * K]
        zt[b * (K + 1) + K] = store(g.normal(0, 2.0, V))
    unif = (g.integers(0, 1 << 24, (B, K + 1)) * 2.0 ** -24).astype(np.float32)
    dev = torch.device("cuda:0")
    dd, td = Hn.to_device(zd, dtype, dev), Hn.to_device(zt, dtype, dev)
    dr = torch.from_numpy(drafted.reshape(-1)).to(dev)
    ud = torch.from_numpy(unif.reshape(-1)).to(dev)
    off = torch.from_numpy((np.arange(B + 1) * (K + 1)).astype(np.int32)).to(dev)
    kd = torch.full((B,), K, dtype=torch.int32, device=dev)
    for mode in (O.MODE_STANDARD, O.MODE_CM, O.MODE_GREEDY):
        row_shape(conf_block)
        st = cmsd.cmsd_confidence(dd)
        row_shape(256)
        n_acc, nxt, ts = cmsd.cmsd_verify(dd, st, td, off, kd, dr, ud, batch=B, k_max=K, mode=mode)
        lp = cmsd.cmsd_logit_pass(dd, td, dr, ud, batch=B, k_max=K, mode=mode, **Hn.PARAMS)
        torch.cuda.synchronize()
        t = Hn.Tally()
        for outs in ((n_acc.cpu().numpy(), nxt.cpu().numpy(), Hn.tstats_np(ts)),
                     (lp["n_accepted"].cpu().numpy(), lp["next_token"].cpu().numpy(),
                      Hn.tstats_np(lp["target_stats"]))):
            na, nx, tsn = outs
            assert na.tolist() == cs, (mode, na.tolist(), cs)
            for b in range(B):
                zdr = [Hn.decode(zd[b * K + i], dtype) for i in range(K)]
                ztr = [Hn.decode(zt[b * (K + 1) + i], dtype) for i in range(K + 1)]
                C = [Hn.oracle_conf(z, V) for z in zdr]
                Hn.check_sequence(t, b, ztr, zdr, drafted[b], unif[b], C, K, mode, Hn.PARAMS, tsn, b * (K + 1),
                                  int(na[b]), int(nx[b]))
                if cs[b] < K and mode != O.MODE_GREEDY:
                    # the final token carries mass in the rejecting row
                    assert ztr[cs[b]][int(nx[b])] > -np.inf
        t.assert_ok()
