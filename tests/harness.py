"""Shared helpers of the GPU parity tests: upload a workload, run the HIP path
through the C ABI, and compare with the oracle under the slack rule (a decision
that differs from the oracle is an allowed, counted exception only when its
oracle slack is below SLACK).  The comparison rules themselves are in
tests/parity.py (numpy only)."""
from __future__ import annotations

import numpy as np
import torch

import workloads as W
from oracle import cmsd_oracle as O  # noqa: F401  (re-exported for the tests)
from tests.parity import (PARAMS, REL, SLACK, Tally, acc_allowed, check_row_stats, check_sequence,  # noqa: F401
                          close_rel, decode, f32, oracle_conf, stats_fields, tstats_fields)


def to_device(stored: np.ndarray, dtype: str, dev) -> torch.Tensor:
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(stored, dtype=np.float32)).to(dev)
    return torch.from_numpy(np.ascontiguousarray(stored).view(np.int16)).to(dev).view(torch.bfloat16)


def stats_np(stats: torch.Tensor) -> dict:
    s = stats.detach().cpu()
    return stats_fields(s.numpy(), s.view(torch.int32).numpy())


def tstats_np(ts: torch.Tensor) -> dict:
    s = ts.detach().cpu()
    return tstats_fields(s.numpy(), s.view(torch.int32).numpy())


# ----------------------------------------------------------------------------- workloads on the device
_CACHE: dict = {}


def workload(name: str, seed: int = 0) -> dict:
    """Host arrays of a workload plus device copies (``*_dev``); at most two cached."""
    key = (name, seed)
    if key in _CACHE:
        d = _CACHE.pop(key)
        _CACHE[key] = d
        return d
    while len(_CACHE) >= 2:
        _CACHE.pop(next(iter(_CACHE)))
    cfg = W.CONFIGS[name]
    d = W.generate(cfg, seed)
    dev = torch.device("cuda:0")
    d["draft_dev"] = to_device(d["draft"], cfg.dtype, dev)
    d["target_dev"] = to_device(d["target"], cfg.dtype, dev)
    d["drafted_dev"] = torch.from_numpy(np.ascontiguousarray(d["drafted"]).reshape(-1)).to(dev)
    d["unif_dev"] = torch.from_numpy(np.ascontiguousarray(d["uniforms"]).reshape(-1)).to(dev)
    _CACHE[key] = d
    return d
