"""One decoding iteration of the logit pass: confidence -> draft length -> verify.

``LogitPass`` preallocates every output once, then ``run`` enqueues the three C
entry points on one stream (no host synchronisation, no allocation), so it can be
timed or captured as is.  Only marshalling happens here.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import cmsd


@dataclass
class Params:
    lambdas: tuple = (1 / 3, 1 / 3, 1 / 3)
    beta_margin: float = 1.0
    k_min: int = 1
    alpha: float = 1.0
    mode: int = cmsd.CMSD_MODE_CM
    top_beta: int = 3
    tau_base: float = 0.1
    gamma: float = 1.0

    # The ablation settings of the paper's Table III, as parameter presets
    # (everything else as given): a fixed draft length, a fixed threshold, both
    # fixed, or a single confidence signal.
    def fixed_k(self, k_max: int) -> "Params":
        return Params(**{**self.__dict__, "k_min": k_max})

    def fixed_tau(self) -> "Params":
        return Params(**{**self.__dict__, "gamma": 0.0})

    def fixed_k_and_tau(self, k_max: int) -> "Params":
        return Params(**{**self.__dict__, "k_min": k_max, "gamma": 0.0})

    def entropy_only(self) -> "Params":
        return Params(**{**self.__dict__, "lambdas": (1.0, 0.0, 0.0)})

    def margin_only(self) -> "Params":
        return Params(**{**self.__dict__, "lambdas": (0.0, 1.0, 0.0)})

    def softmax_only(self) -> "Params":
        return Params(**{**self.__dict__, "lambdas": (0.0, 0.0, 1.0)})


class LogitPass:
    """Buffers and calls for B sequences of k_max drafted positions over vocab V.

    ``dense=True``: the verifier scored all k_max+1 positions of every sequence, so
    verify runs with k_b = k_max and offsets b*(k_max+1) (the draft lengths are still
    computed and returned).  ``dense=False``: verify consumes the device-computed
    k_b and offsets; the caller supplies target rows and uniforms packed by those
    offsets (``target_rows`` allocated rows, at most B*(k_max+1)).
    """

    def __init__(self, B: int, k_max: int, V: int, device, params: Params | None = None,
                 dense: bool = True, target_rows: int | None = None):
        self.B, self.k_max, self.V = B, k_max, V
        self.p = params or Params()
        self.dense = dense
        dev = torch.device(device)
        self.target_rows = target_rows or B * (k_max + 1)
        self.stats = torch.empty((B * k_max, 8), dtype=torch.float32, device=dev)
        self.k = torch.empty(B, dtype=torch.int32, device=dev)
        self.off = torch.empty(B + 1, dtype=torch.int32, device=dev)
        self.k_dense = torch.full((B,), k_max, dtype=torch.int32, device=dev)
        self.off_dense = (torch.arange(B + 1, dtype=torch.int32, device=dev) * (k_max + 1)).contiguous()
        self.tstats = torch.empty((self.target_rows, 8), dtype=torch.float32, device=dev)
        self.n_acc = torch.empty(B, dtype=torch.int32, device=dev)
        self.next_tok = torch.empty(B, dtype=torch.int32, device=dev)
        self.ws = cmsd.verify_workspace(B, k_max, V, dev)

    def confidence(self, draft: torch.Tensor, stream=None) -> None:
        cmsd.cmsd_confidence(draft, self.stats, lambdas=self.p.lambdas, beta_margin=self.p.beta_margin,
                             stream=stream)

    def draft_len(self, stream=None) -> None:
        cmsd.cmsd_draft_len(self.stats, self.B, k_min=self.p.k_min, k_max=self.k_max, alpha=self.p.alpha,
                            draft_len=self.k, target_offsets=self.off, stream=stream)

    def verify(self, draft: torch.Tensor, target: torch.Tensor, drafted: torch.Tensor, uniforms: torch.Tensor,
               stream=None) -> None:
        k, off = (self.k_dense, self.off_dense) if self.dense else (self.k, self.off)
        cmsd.cmsd_verify(draft, self.stats, target, off, k, drafted, uniforms, batch=self.B, k_max=self.k_max,
                         mode=self.p.mode, top_beta=self.p.top_beta, tau_base=self.p.tau_base,
                         gamma=self.p.gamma, target_stats=self.tstats, n_accepted=self.n_acc,
                         next_token=self.next_tok, workspace=self.ws, stream=stream)

    def run(self, draft, target, drafted, uniforms, stream=None) -> None:
        """confidence + draft_len + verify, enqueued on ``stream``."""
        self.confidence(draft, stream)
        self.draft_len(stream)
        self.verify(draft, target, drafted, uniforms, stream)

    def logit_pass(self, draft, target, drafted, uniforms, stream=None, row_events=None, adaptive=False) -> None:
        """The same iteration as one cmsd_logit_pass call (dense target layout only):
        drafter and target rows in one row pass, then the final-token pass.
        ``adaptive``: verify only the first k_b drafts of each sequence."""
        if not self.dense:
            raise ValueError("cmsd_logit_pass takes the dense target layout; this LogitPass is packed")
        p = self.p
        cmsd.cmsd_logit_pass(draft, target, drafted, uniforms, batch=self.B, k_max=self.k_max, lambdas=p.lambdas,
                             beta_margin=p.beta_margin, k_min=p.k_min, alpha=p.alpha, mode=p.mode,
                             top_beta=p.top_beta, tau_base=p.tau_base, gamma=p.gamma, adaptive=adaptive,
                             draft_stats=self.stats, draft_len=self.k, target_stats=self.tstats,
                             n_accepted=self.n_acc, next_token=self.next_tok, workspace=self.ws,
                             row_events=row_events, stream=stream)

    def logit_pass_fused(self, draft, target, drafted, uniforms, stream=None, adaptive=False) -> None:
        """The same iteration as one cmsd_logit_pass_fused call: a single launch, for
        small batches (dense target layout only).  Its zero-filled workspace is
        allocated on first use and kept."""
        if not self.dense:
            raise ValueError("cmsd_logit_pass_fused takes the dense target layout; this LogitPass is packed")
        if getattr(self, "fws", None) is None:
            self.fws = cmsd.fused_workspace(self.B, self.k_max, self.V, self.stats.device)
        p = self.p
        cmsd.cmsd_logit_pass_fused(draft, target, drafted, uniforms, batch=self.B, k_max=self.k_max,
                                   lambdas=p.lambdas, beta_margin=p.beta_margin, k_min=p.k_min, alpha=p.alpha,
                                   mode=p.mode, top_beta=p.top_beta, tau_base=p.tau_base, gamma=p.gamma,
                                   adaptive=adaptive, draft_stats=self.stats, draft_len=self.k,
                                   target_stats=self.tstats, n_accepted=self.n_acc, next_token=self.next_tok,
                                   workspace=self.fws, stream=stream)
