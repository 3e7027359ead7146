"""Speculative decoding loop around the logit pass, on synthetic random-weight models.

The loop follows Sec. III.A with the confidence machinery of Sec. III.B: the drafter
proposes k_max tokens (exact softmax samples, or its top token in GREEDY mode), the
drafter-row confidences choose each sequence's draft length k_b, the target scores
the drafts, and verification keeps the accepted prefix plus one token.  Every step
of the method runs in the library's kernels (``cmsd_draft_sample``,
``cmsd_confidence``, ``cmsd_draft_len``, ``cmsd_verify``); this module only runs the
two models and keeps the token buffers.

The models are small causal transformers with seeded random weights: there are no
trained weights here.  The drafter is the target with seeded weight noise, so the
two agree often and the drafter's confidence tracks how often (the regime the
method targets).  ``python -m paper_2508_15371_amd.decode`` prints tokens per
iteration, draft length and rollback frequency for the Table III settings.
"""
from __future__ import annotations

import copy
import math
from dataclasses import dataclass, field

import torch

from . import cmsd, pipeline


class TinyLM(torch.nn.Module):
    """Causal transformer LM with seeded random weights (pre-norm, GELU MLP); the
    logits are multiplied by ``scale`` so rows range from flat to peaked."""

    def __init__(self, vocab: int, d: int = 256, layers: int = 2, heads: int = 4, max_len: int = 512,
                 seed: int = 0, scale: float = 5.0):
        super().__init__()
        g = torch.Generator().manual_seed(seed)

        def w(*shape, std):
            return torch.nn.Parameter(torch.randn(*shape, generator=g) * std)

        self.vocab, self.d, self.heads, self.scale = vocab, d, heads, scale
        self.emb = w(vocab, d, std=1.0)
        self.pos = w(max_len, d, std=0.5)
        self.layers = torch.nn.ModuleList()
        for _ in range(layers):
            blk = torch.nn.ParameterDict({
                "qkv": w(d, 3 * d, std=d ** -0.5), "o": w(d, d, std=d ** -0.5),
                "up": w(d, 4 * d, std=d ** -0.5), "down": w(4 * d, d, std=(4 * d) ** -0.5)})
            self.layers.append(blk)
        self.out = w(d, vocab, std=d ** -0.5)

    def perturbed(self, noise: float, seed: int) -> "TinyLM":
        """A copy with N(0, (noise * std(w))^2) added to every weight tensor."""
        m = copy.deepcopy(self)
        g = torch.Generator().manual_seed(seed)
        with torch.no_grad():
            for p in m.parameters():
                p.add_(torch.randn(p.shape, generator=g).to(p.device) * (noise * float(p.std())))
        return m

    @torch.no_grad()
    def forward(self, tok: torch.Tensor) -> torch.Tensor:
        """tok [B, T] int64 -> logits [B, T, V] float32 (causal)."""
        B, T = tok.shape
        x = self.emb[tok] + self.pos[:T]
        mask = torch.full((T, T), float("-inf"), device=tok.device).triu(1)
        H, dh = self.heads, self.d // self.heads
        for blk in self.layers:
            h = torch.nn.functional.layer_norm(x, (self.d,))
            q, k, v = (h @ blk["qkv"]).split(self.d, -1)
            q = q.view(B, T, H, dh).transpose(1, 2).contiguous()
            kt = k.view(B, T, H, dh).permute(0, 2, 3, 1).contiguous()
            v = v.view(B, T, H, dh).transpose(1, 2).contiguous()
            a = torch.softmax(torch.matmul(q, kt) / math.sqrt(dh) + mask, -1)
            x = x + torch.matmul(a, v).transpose(1, 2).reshape(B, T, self.d) @ blk["o"]
            h = torch.nn.functional.layer_norm(x, (self.d,))
            x = x + torch.nn.functional.gelu(h @ blk["up"]) @ blk["down"]
        h = torch.nn.functional.layer_norm(x, (self.d,))
        return (self.scale * (h @ self.out)).float()


@dataclass
class DecodeStats:
    iterations: int = 0
    tokens: int = 0          # tokens appended (accepted drafts + one per iteration and sequence)
    drafted: int = 0         # sum of k_b
    accepted: int = 0        # sum of n_acc
    rollbacks: int = 0       # sequence-iterations that rejected a draft
    seq_iters: int = 0
    k_hist: list = field(default_factory=list)

    def row(self) -> dict:
        return {"tokens_per_iteration": self.tokens / max(1, self.seq_iters),
                "mean_draft_len": self.drafted / max(1, self.seq_iters),
                "acceptance": self.accepted / max(1, self.drafted),
                "rollback_frequency": self.rollbacks / max(1, self.seq_iters)}


class SpeculativeDecoder:
    """B sequences decoded together; drafter and target share the vocabulary."""

    def __init__(self, target: TinyLM, drafter: TinyLM, B: int, k_max: int, params: pipeline.Params,
                 device, seed: int = 0, max_len: int = 512):
        self.t, self.d = target, drafter
        self.B, self.K, self.V = B, k_max, target.vocab
        self.p = params
        self.dev = torch.device(device)
        self.greedy = params.mode == cmsd.CMSD_MODE_GREEDY
        self.lp = pipeline.LogitPass(B, k_max, self.V, self.dev, params, dense=False, target_rows=B * (k_max + 1))
        self.dl = torch.empty((B, k_max, self.V), dtype=torch.float32, device=self.dev)
        self.drafted = torch.empty((B, k_max), dtype=torch.int32, device=self.dev)
        self.st_step = torch.empty((B, 8), dtype=torch.float32, device=self.dev)
        self.draw = torch.empty(B, dtype=torch.int32, device=self.dev)
        self.ws_draft = torch.empty(max(1, (cmsd.cmsd_draft_sample_workspace_bytes(B, self.V) + 7) // 8),
                                    dtype=torch.float64, device=self.dev)
        self.gen = torch.Generator(device=self.dev).manual_seed(seed)
        self.max_len = max_len
        self.stats = DecodeStats()

    def _uniform(self, n: int) -> torch.Tensor:
        return torch.rand(n, generator=self.gen, device=self.dev, dtype=torch.float32)

    def step(self, tok: torch.Tensor, lens: torch.Tensor, active: torch.Tensor | None = None,
             record: list | None = None) -> None:
        """One iteration on the padded token buffer tok [B, cap] (valid prefix lens[b]);
        sequences where ``active`` is False are decoded but not advanced or counted.
        ``record``: if a list, a host copy of the iteration's inputs and outputs of
        the library calls is appended to it (for checking an iteration elsewhere)."""
        B, K = self.B, self.K
        draft_u = []
        ar = torch.arange(B, device=self.dev)
        lmax = int(lens.max())
        assert lmax + K + 1 <= tok.shape[1] and lmax + K <= self.max_len
        # drafting: k_max drafter positions per sequence
        for i in range(K):
            z = self.d(tok[:, :lmax + i])
            self.dl[:, i] = z[ar, lens + i - 1]
            rows = self.dl[:, i]
            cmsd.cmsd_confidence(rows, self.st_step, lambdas=self.p.lambdas, beta_margin=self.p.beta_margin)
            if self.greedy:
                self.draw.copy_(self.st_step.view(torch.int32)[:, 6])     # the drafter's top token
            else:
                u = self._uniform(B)
                draft_u.append(u)
                cmsd.cmsd_draft_sample(rows, self.st_step, u, drafted=self.draw, workspace=self.ws_draft)
            self.drafted[:, i] = self.draw
            tok[ar, lens + i] = self.draw.long()
            self.lp.stats.view(B, K, 8)[:, i] = self.st_step
        # confidence -> draft lengths and packed offsets
        self.lp.draft_len()
        # target scores every drafted position; packed rows: b's rows 0..k_b
        zt = self.t(tok[:, :lmax + K])
        pos = (lens.view(B, 1) - 1 + torch.arange(K + 1, device=self.dev).view(1, K + 1)).clamp(max=lmax + K - 1)
        dense = zt[ar.view(B, 1), pos]                                   # [B, K+1, V]
        R = B * (K + 1)
        p = torch.arange(R, device=self.dev)
        off = self.lp.off.long()
        b = torch.searchsorted(off[1:].contiguous(), p, right=True).clamp(max=B - 1)
        i = (p - off[b]).clamp(min=0, max=K)
        target = dense.reshape(R, self.V).index_select(0, b * (K + 1) + i)
        unif = None if self.greedy else self._uniform(R)
        self.lp.verify(self.dl.view(B * K, self.V), target, self.drafted.view(-1), unif)
        n_acc = self.lp.n_acc.long()
        nxt = self.lp.next_tok.long()
        k = self.lp.k.long()
        if record is not None:
            record.append({"draft": self.dl.cpu(), "draft_u": torch.stack(draft_u, 1).cpu() if draft_u else None,
                           "drafted": self.drafted.cpu(), "stats": self.lp.stats.cpu(), "k": self.lp.k.cpu(),
                           "off": self.lp.off.cpu(), "target": target.cpu(),
                           "unif": None if unif is None else unif.cpu(), "tstats": self.lp.tstats.cpu(),
                           "n_acc": self.lp.n_acc.cpu(), "next": self.lp.next_tok.cpu()})
        if bool((n_acc < 0).any()):
            raise RuntimeError("cmsd_verify reported an invalid sequence")
        if active is None:
            active = torch.ones(B, dtype=torch.bool, device=self.dev)
        tok[ar, lens + n_acc] = torch.where(active, nxt, tok[ar, lens + n_acc])
        lens += torch.where(active, n_acc + 1, torch.zeros_like(n_acc))
        s = self.stats
        a = active.long()
        s.iterations += 1
        s.seq_iters += int(a.sum())
        s.tokens += int(((n_acc + 1) * a).sum())
        s.drafted += int((k * a).sum())
        s.accepted += int((n_acc * a).sum())
        s.rollbacks += int(((n_acc < k).long() * a).sum())
        s.k_hist.extend(k[active].tolist())

    def generate(self, prompt: torch.Tensor, n_new: int) -> list:
        """Decode until every sequence has at least n_new new tokens; returns each
        sequence's first n_new new tokens."""
        B, L0 = prompt.shape
        cap = L0 + n_new + 2 * self.K + 2
        tok = torch.zeros((B, cap), dtype=torch.long, device=self.dev)
        tok[:, :L0] = prompt
        lens = torch.full((B,), L0, dtype=torch.long, device=self.dev)
        while int(lens.min()) < L0 + n_new:
            self.step(tok, lens, lens < L0 + n_new)
        return [tok[b, L0:L0 + n_new].tolist() for b in range(B)]


def greedy_reference(target: TinyLM, prompt: torch.Tensor, n_new: int) -> tuple[list, list]:
    """The target's own greedy decode (lowest index among equal maxima) and, per
    step, the gap between its two largest logits."""
    tok = prompt.clone()
    gaps = []
    for _ in range(n_new):
        z = target(tok)[:, -1].double()
        top2 = torch.topk(z, 2, -1).values
        gaps.append((top2[:, 0] - top2[:, 1]).tolist())
        tok = torch.cat([tok, torch.argmax(z, -1, keepdim=True)], 1)
    return [tok[b, prompt.shape[1]:].tolist() for b in range(prompt.shape[0])], gaps


def _report(device="cuda:0", B=16, k_max=8, V=32000, n_new=96, seed=0, noise=0.1) -> list:
    target = TinyLM(V, seed=seed + 1).to(device)
    drafter = target.perturbed(noise, seed + 2).to(device)
    prompt = torch.randint(0, V, (B, 16), generator=torch.Generator().manual_seed(seed)).to(device)
    base = pipeline.Params()
    settings = [
        ("CM, adaptive k and tau", base),
        ("STANDARD, adaptive k", pipeline.Params(**{**base.__dict__, "mode": cmsd.CMSD_MODE_STANDARD})),
        ("CM, fixed k = k_max", base.fixed_k(k_max)),
        ("CM, fixed tau", base.fixed_tau()),
        ("CM, fixed k and tau", base.fixed_k_and_tau(k_max)),
        ("CM, entropy only", base.entropy_only()),
        ("CM, logit margin only", base.margin_only()),
        ("CM, softmax margin only", base.softmax_only()),
        ("GREEDY, gate off (exact match)", pipeline.Params(**{**base.__dict__, "mode": cmsd.CMSD_MODE_GREEDY,
                                                               "top_beta": 0})),
        ("GREEDY, adaptive gate", pipeline.Params(**{**base.__dict__, "mode": cmsd.CMSD_MODE_GREEDY})),
    ]
    rows = []
    for name, prm in settings:
        dec = SpeculativeDecoder(target, drafter, B, k_max, prm, device, seed=seed)
        dec.generate(prompt, n_new)
        r = dec.stats.row()
        r["setting"] = name
        rows.append(r)
    return rows


if __name__ == "__main__":
    rows = _report()
    print(f"{'setting':34s} {'tok/iter':>8s} {'mean k':>7s} {'accept':>7s} {'rollback':>8s}")
    for r in rows:
        print(f"{r['setting']:34s} {r['tokens_per_iteration']:8.3f} {r['mean_draft_len']:7.2f} "
              f"{r['acceptance']:7.3f} {r['rollback_frequency']:8.3f}")
