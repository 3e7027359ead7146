"""GPU parity of cmsd_draft_sample (one softmax sample per drafter row) against the
oracle's inverse-CDF draw, through the C ABI."""
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


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V", [2, 7, 1000, 32000, 50257, 128259, 600011])
def test_draft_sample_rows(cm, dtype, V):
    g = np.random.default_rng(V + (7 if dtype == "bf16" else 0))
    n = 24
    z = np.stack([g.normal(0, float(g.uniform(0.2, 6)), V) for _ in range(n)]).astype(np.float32)
    for r in range(0, n, 5):
        m = g.random(V) < 0.3
        m[int(np.argmax(z[r]))] = False
        z[r][m] = -np.inf
    stored = z if dtype == "f32" else W.bf16_bits_from_f32(z)
    u = (g.integers(0, 1 << 24, n) * 2.0 ** -24).astype(np.float32)
    u[0], u[1] = 0.0, np.float32(1.0 - 2.0 ** -24)
    dev = torch.device("cuda:0")
    x = Hn.to_device(stored, dtype, dev)
    st = cm.cmsd_confidence(x)
    y = cm.cmsd_draft_sample(x, st, torch.from_numpy(u).to(dev))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    t = Hn.Tally()
    for r in range(n):
        want, slack = O.draft_sample(Hn.decode(stored[r], dtype), float(u[r]))
        t.decision(f"y[{r}]", int(y[r]), want, slack)
    t.assert_ok()


def test_draft_sample_workload_rows(cm):
    d = Hn.workload("c3", 0)
    g = np.random.default_rng(3)
    n = d["draft"].shape[0]
    u = (g.integers(0, 1 << 24, n) * 2.0 ** -24).astype(np.float32)
    dev = torch.device("cuda:0")
    st = cm.cmsd_confidence(d["draft_dev"])
    y = cm.cmsd_draft_sample(d["draft_dev"], st, torch.from_numpy(u).to(dev))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    t = Hn.Tally()
    for r in g.choice(n, 48, replace=False):
        want, slack = O.draft_sample(Hn.decode(d["draft"][r], "bf16"), float(u[r]))
        t.decision(f"y[{r}]", int(y[r]), want, slack)
    t.assert_ok()


@pytest.mark.parametrize("seed", range(8))
def test_draft_sample_random_rows(cm, seed):
    # seeded random problems: vocabulary 2..300000 (log-uniform), 1..40 rows of random
    # scale, padded strides, per-row masks of random density, uniforms at both ends of
    # [0, 1) among them; every sample against the oracle's inverse CDF
    g = np.random.default_rng(5000 + seed)
    V = int(round(math.exp(g.uniform(math.log(2), math.log(300000)))))
    n, pad = int(g.integers(1, 41)), int(g.integers(0, 6))
    dtype = ("f32", "bf16")[int(g.integers(2))]
    frac = (0.0, 0.05, 0.5, 0.95)[int(g.integers(4))]
    print(f"V={V} n={n} pad={pad} {dtype} mask={frac}", flush=True)
    z = np.stack([g.normal(0, float(g.uniform(0.2, 8)), V) for _ in range(n)]).astype(np.float32)
    if frac > 0.0:
        m = g.random(z.shape) < frac
        m[np.arange(n), g.integers(0, V, n)] = False
        z[m] = -np.inf
    stored = z if dtype == "f32" else W.bf16_bits_from_f32(z)
    buf = np.zeros((n, V + pad), dtype=stored.dtype)
    buf[:, :V] = stored
    u = (g.integers(0, 1 << 24, n) * 2.0 ** -24).astype(np.float32)
    u[0] = 0.0
    u[-1] = np.float32(1.0 - 2.0 ** -24)
    dev = torch.device("cuda:0")
    x = Hn.to_device(buf, dtype, dev)[:, :V]
    st = cm.cmsd_confidence(x)
    y = cm.cmsd_draft_sample(x, st, torch.from_numpy(u).to(dev))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    t = Hn.Tally()
    for r in range(n):
        want, slack = O.draft_sample(Hn.decode(stored[r], dtype), float(u[r]))
        t.decision(f"y[{r}]", int(y[r]), want, slack)
    t.assert_ok()
