"""Seeded synthetic inputs for the confidence / draft-length / verify pass.

This module is shared by the CPU oracle's tests, the GPU parity tests and the
benchmark.  It only draws random numbers and rounds them to the storage dtype;
it computes none of the quantities the method defines (no softmax, entropy,
margin, confidence, draft length, acceptance or residual sampling).

Every random stream is keyed by ``SeedSequence([config_id, seed, stream, index])``
so that any single row can be regenerated on its own (the parity tests use this
to check sampled rows of the full-size workloads without materialising them on
the host twice), and so that rows can be generated in parallel threads.

Workloads (the paper evaluates on WMT'14/'16 translation and CNN/DailyMail with
trained Transformer/BART models, Section IV.A; neither the datasets nor the
weights are available, so these seeded logit distributions stand in for the
drafter and verifier outputs):

* ``tiny`` : B=1, k=4, V=1024, fp32.  Drafter row i ~ N(0, s_i^2) with s cycling
  (0.5, 2, 8, 0.5); target rows 0..3 = drafter + N(0, 0.5^2); target row 4 ~
  N(0, 2^2).  Drafted ids are the drafter argmax (lowest index on ties).
* ``c2``   : B=8, k_max=8, V=32000, bf16.  Row scale s log-uniform in [0.3, 10]
  times N(0,1).  Target = d*(1+N(0,0.1^2)) + N(0,0.3^2) per element; the bonus
  row is a fresh s*N(0,1) row.  Drafts sampled from the drafter softmax.
* ``c3``   : B=64, k_max=8, V=50257, bf16.  Zipf-peaked rows
  z_v = a*(-1.1*ln rank_pi(v)) + N(0,0.2^2), a ~ U[0.5,3] per row, pi a seeded
  permutation per row.  Target rows reuse pi and a with fresh noise, except
  round(0.2*R_t) seeded rows that use an independent permutation.
* ``c4``   : B=256, k_max=16, V=128256, bf16.  Drafter rows split by a seeded
  permutation into near-one-hot (N(0,0.3^2) + 15 at one seeded index), Zipf
  (as c3) and flat N(0,0.3^2) thirds.  Target = drafter + N(0,0.5^2); the bonus
  row is a fresh row of the regime of the sequence's last drafter row.
* ``c5``   : ragged, B=512, k_max=16, V=32000, bf16.  Drafter rows s*N(0,1), s
  log-uniform in [0.3, 10].  Target rows i < k_b = drafter + N(0,0.5^2); the
  row at k_b is a fresh s'*N(0,1) row.  Draft lengths k_b come from the
  draft-length step on the device, so targets and uniforms are produced padded
  ``[B, k_max+1, V]`` (bonus row stored at slot k_max) and packed afterwards.
* ``v152k``: a sweep point, not one of the five: B=64, k_max=8, V=152064 (the top
  of the metric's vocabulary range), bf16, with c2's row recipe.
* ``c4f``  : c4's recipe stored in fp32 (its own seeded streams, no bf16 rounding):
  the headline shape for the fp32 row kernels.
* ``c5m``  : c5 with masked logits: every drafter row and the target row of the same
  position set -inf on one seeded mask of the vocabulary (the last 128 tokens, as
  padding of a vocabulary rounded up, plus 3 % of the others at random, as a decoding
  constraint); each bonus row has a mask of its own.  Drafts never land on a masked
  token (they are softmax samples).

Uniforms are ``randint(0, 2^24) * 2^-24`` as fp32: exactly representable and
strictly below 1.  Drafted ids (except ``tiny``) are exact samples from the
softmax of the stored drafter logits, drawn with the Gumbel-max construction
(argmax of logit + Gumbel noise) from their own seeded uniform stream.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

__all__ = [
    "CONFIGS", "Config", "bf16_bits_from_f32", "f32_from_bf16_bits",
    "draft_row", "target_row", "drafted_id", "uniform", "generate",
    "pack_ragged",
]

# stream ids (third SeedSequence word)
_S_DRAFT_SCALE = 1
_S_DRAFT_ROW = 2
_S_TARGET_ROW = 3
_S_BONUS_ROW = 4
_S_GUMBEL = 5
_S_UNIFORM = 6
_S_REGIME = 7
_S_INDEP = 8
_S_MASK = 9
_S_BONUS_MASK = 10


@dataclass(frozen=True)
class Config:
    name: str
    cid: int
    B: int
    k_max: int
    V: int
    dtype: str          # "f32" or "bf16"
    ragged: bool = False
    style: str = ""     # row recipe of another config (a sweep point), else the config's own
    masked: bool = False  # -inf on a seeded mask per position (see c5m)

    @property
    def kind(self) -> str:
        return self.style or self.name

    @property
    def draft_rows(self) -> int:
        return self.B * self.k_max

    @property
    def dense_target_rows(self) -> int:
        return self.B * (self.k_max + 1)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


CONFIGS = {
    "tiny": Config("tiny", 0, 1, 4, 1024, "f32"),
    "c2": Config("c2", 1, 8, 8, 32000, "bf16"),
    "c3": Config("c3", 2, 64, 8, 50257, "bf16"),
    "c4": Config("c4", 3, 256, 16, 128256, "bf16"),
    "c5": Config("c5", 4, 512, 16, 32000, "bf16", ragged=True),
    # sweep point at the top of the metric's vocabulary range, with c2's row recipe
    "v152k": Config("v152k", 5, 64, 8, 152064, "bf16", style="c2"),
    # one sequence (single-stream decoding latency), with c2's row recipe
    "b1": Config("b1", 6, 1, 8, 32000, "bf16", style="c2"),
    # c5 with masked logits (vocabulary padding and a decoding constraint)
    "c5m": Config("c5m", 7, 512, 16, 32000, "bf16", ragged=True, style="c5", masked=True),
    # c4's rows in fp32 (the fp32 row kernels at the headline shape)
    "c4f": Config("c4f", 8, 256, 16, 128256, "f32", style="c4"),
}

_MASK_TAIL = 128       # masked tokens at the end of the vocabulary
_MASK_FRAC = 0.03      # masked share of the other tokens


def _mask(cfg: Config, seed: int, stream: int, index: int) -> np.ndarray:
    """Boolean [V] mask of a masked config: the last _MASK_TAIL tokens and a seeded
    _MASK_FRAC of the others."""
    V = cfg.V
    g = _rng(cfg, seed, stream, index)
    m = g.random(V) < _MASK_FRAC
    m[V - _MASK_TAIL:] = True
    return m


def _masked(cfg: Config, z: np.ndarray, seed: int, stream: int, index: int) -> np.ndarray:
    if not cfg.masked:
        return z
    z = np.array(z, dtype=np.float64)
    z[_mask(cfg, seed, stream, index)] = -np.inf
    return z


def _rng(cfg: Config, seed: int, stream: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.cid, seed, stream, index])))


# ----------------------------------------------------------------------------- storage rounding
def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return the raw uint16 bits.

    Inputs here are finite or -inf (masked logits), so no NaN special case is needed.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """Widen raw bfloat16 bits to float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _store(cfg: Config, x: np.ndarray) -> np.ndarray:
    """Round a float array to the config's storage dtype (uint16 bits for bf16, float32 for f32)."""
    x32 = np.asarray(x, dtype=np.float32)
    return x32 if cfg.dtype == "f32" else bf16_bits_from_f32(x32)


def _stored_as_f32(cfg: Config, stored: np.ndarray) -> np.ndarray:
    return stored if cfg.dtype == "f32" else f32_from_bf16_bits(stored)


# ----------------------------------------------------------------------------- row recipes
_LOGRANK: dict[int, np.ndarray] = {}


def _log_rank(V: int) -> np.ndarray:
    t = _LOGRANK.get(V)
    if t is None:
        t = np.log(np.arange(1, V + 1, dtype=np.float64))
        _LOGRANK[V] = t
    return t


def _zipf_row(V: int, perm: np.ndarray, a: float, noise: np.ndarray) -> np.ndarray:
    # element v has rank perm[v] + 1
    return a * (-1.1 * _log_rank(V)[perm]) + noise


def _c4_regime(cfg: Config, seed: int, row: int) -> int:
    """0 = near-one-hot, 1 = Zipf, 2 = flat; exact thirds over a seeded permutation of the rows."""
    perm = _c4_perm_cache(cfg, seed)
    pos = int(perm[row])
    n = cfg.draft_rows
    return 0 if pos < n // 3 else (1 if pos < 2 * (n // 3) else 2)


_PERM_CACHE: dict[tuple, np.ndarray] = {}


def _c4_perm_cache(cfg: Config, seed: int) -> np.ndarray:
    key = (cfg.cid, seed)
    p = _PERM_CACHE.get(key)
    if p is None:
        order = _rng(cfg, seed, _S_REGIME, 0).permutation(cfg.draft_rows)
        p = np.empty_like(order)
        p[order] = np.arange(cfg.draft_rows)   # p[row] = position of row in the shuffled order
        _PERM_CACHE[key] = p
    return p


def _c3_indep_rows(cfg: Config, seed: int) -> set:
    key = ("indep", cfg.cid, seed)
    s = _PERM_CACHE.get(key)
    if s is None:
        n = cfg.dense_target_rows
        n_indep = int(round(0.2 * n))
        s = set(_rng(cfg, seed, _S_INDEP, 0).choice(n, size=n_indep, replace=False).tolist())
        _PERM_CACHE[key] = s
    return s


def _draft_row_f64(cfg: Config, seed: int, row: int) -> np.ndarray:
    """Unrounded drafter row ``row`` (= b*k_max + i) as float64."""
    V = cfg.V
    g = _rng(cfg, seed, _S_DRAFT_ROW, row)
    if cfg.kind == "tiny":
        s = (0.5, 2.0, 8.0, 0.5)[row % 4]
        return s * g.standard_normal(V)
    if cfg.kind in ("c2", "c5"):
        s = math.exp(g.uniform(math.log(0.3), math.log(10.0)))
        return s * g.standard_normal(V, dtype=np.float32).astype(np.float64)
    if cfg.kind == "c3":
        a = g.uniform(0.5, 3.0)
        perm = g.permutation(V)
        return _zipf_row(V, perm, a, 0.2 * g.standard_normal(V, dtype=np.float32).astype(np.float64))
    if cfg.kind == "c4":
        reg = _c4_regime(cfg, seed, row)
        return _c4_regime_row(V, reg, g)
    raise KeyError(cfg.kind)


def _c4_regime_row(V: int, reg: int, g: np.random.Generator) -> np.ndarray:
    if reg == 0:
        z = 0.3 * g.standard_normal(V, dtype=np.float32).astype(np.float64)
        z[int(g.integers(0, V))] += 15.0
        return z
    if reg == 1:
        a = g.uniform(0.5, 3.0)
        perm = g.permutation(V)
        return _zipf_row(V, perm, a, 0.2 * g.standard_normal(V, dtype=np.float32).astype(np.float64))
    return 0.3 * g.standard_normal(V, dtype=np.float32).astype(np.float64)


def draft_row(cfg: Config, seed: int, row: int) -> np.ndarray:
    """Stored drafter row ``row`` (= b*k_max + i): float32 values, or uint16 bf16 bits."""
    return _store(cfg, _masked(cfg, _draft_row_f64(cfg, seed, row), seed, _S_MASK, row))


def _c3_params(cfg: Config, seed: int, row: int):
    """Re-derive (a, perm) of c3 drafter row ``row`` (same stream order as _draft_row_f64)."""
    g = _rng(cfg, seed, _S_DRAFT_ROW, row)
    a = g.uniform(0.5, 3.0)
    perm = g.permutation(cfg.V)
    return a, perm


def target_row(cfg: Config, seed: int, b: int, i: int, draft_stored: np.ndarray | None = None) -> np.ndarray:
    """Stored target row for sequence ``b``, position ``i`` in 0..k_max (masked configs:
    position i < k_max shares drafter row b*k_max+i's mask, the bonus row has its own)."""
    z = _target_row_unmasked(cfg, seed, b, i, draft_stored)
    if not cfg.masked:
        return z
    zf = _stored_as_f32(cfg, z).astype(np.float64)
    K = cfg.k_max
    if i == K:
        zf[_mask(cfg, seed, _S_BONUS_MASK, b)] = -np.inf
    else:
        zf[_mask(cfg, seed, _S_MASK, b * K + i)] = -np.inf
    return _store(cfg, zf)


def _target_row_unmasked(cfg: Config, seed: int, b: int, i: int,
                         draft_stored: np.ndarray | None = None) -> np.ndarray:
    """Stored target row for sequence ``b``, position ``i`` in 0..k_max.

    Position ``k_max`` is the bonus row (for the ragged config it is the row that
    ends up at slot k_b after packing).  ``draft_stored`` may pass the already
    generated stored drafter row (b, i) to avoid regenerating it.
    """
    V, K = cfg.V, cfg.k_max
    bonus = i == K
    if cfg.kind == "tiny":
        g = _rng(cfg, seed, _S_TARGET_ROW, b * (K + 1) + i)
        if bonus:
            return _store(cfg, 2.0 * g.standard_normal(V))
        d = _stored_as_f32(cfg, draft_stored if draft_stored is not None else draft_row(cfg, seed, b * K + i))
        return _store(cfg, d.astype(np.float64) + 0.5 * g.standard_normal(V))
    if bonus:
        g = _rng(cfg, seed, _S_BONUS_ROW, b)
        if cfg.kind in ("c2", "c5"):
            s = math.exp(g.uniform(math.log(0.3), math.log(10.0)))
            return _store(cfg, s * g.standard_normal(V, dtype=np.float32).astype(np.float64))
        if cfg.kind == "c3":
            a = g.uniform(0.5, 3.0)
            perm = g.permutation(V)
            return _store(cfg, _zipf_row(V, perm, a, 0.2 * g.standard_normal(V, dtype=np.float32).astype(np.float64)))
        if cfg.kind == "c4":
            reg = _c4_regime(cfg, seed, b * K + K - 1)
            return _store(cfg, _c4_regime_row(V, reg, g))
        raise KeyError(cfg.kind)
    row = b * K + i
    g = _rng(cfg, seed, _S_TARGET_ROW, b * (K + 1) + i)
    if cfg.kind == "c3":
        a, perm = _c3_params(cfg, seed, row)
        if (b * (K + 1) + i) in _c3_indep_rows(cfg, seed):
            perm = g.permutation(V)
        return _store(cfg, _zipf_row(V, perm, a, 0.2 * g.standard_normal(V, dtype=np.float32).astype(np.float64)))
    d = _stored_as_f32(cfg, draft_stored if draft_stored is not None else draft_row(cfg, seed, row)).astype(np.float64)
    if cfg.kind == "c2":
        n1 = g.standard_normal(V, dtype=np.float32).astype(np.float64)
        n2 = g.standard_normal(V, dtype=np.float32).astype(np.float64)
        return _store(cfg, d * (1.0 + 0.1 * n1) + 0.3 * n2)
    if cfg.kind in ("c4", "c5"):
        return _store(cfg, d + 0.5 * g.standard_normal(V, dtype=np.float32).astype(np.float64))
    raise KeyError(cfg.kind)


def drafted_id(cfg: Config, seed: int, row: int, draft_stored: np.ndarray | None = None) -> int:
    """Drafted token for drafter row ``row``.

    ``tiny``: the argmax of the stored row (lowest index on ties).  Otherwise an
    exact sample from the softmax of the stored logits via Gumbel-max.
    """
    d = draft_stored if draft_stored is not None else draft_row(cfg, seed, row)
    z = _stored_as_f32(cfg, d).astype(np.float64)
    if cfg.kind == "tiny":
        return int(np.argmax(z))
    g = _rng(cfg, seed, _S_GUMBEL, row)
    u = g.random(cfg.V)                      # [0, 1)
    u = np.maximum(u, np.finfo(np.float64).tiny)
    return int(np.argmax(z - np.log(-np.log(u))))


def uniform(cfg: Config, seed: int, b: int) -> np.ndarray:
    """The k_max+1 fp32 uniforms of sequence ``b``: slots 0..k_max-1 for the accept tests of
    positions 0..k_max-1, slot k_max for the final sample (placed at slot k_b after packing)."""
    g = _rng(cfg, seed, _S_UNIFORM, b)
    return (g.integers(0, 1 << 24, size=cfg.k_max + 1).astype(np.float64) * 2.0 ** -24).astype(np.float32)


# ----------------------------------------------------------------------------- bulk generation
def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def generate(cfg: Config | str, seed: int = 0, threads: int | None = None) -> dict:
    """Materialise a whole workload on the host.

    Returns a dict with
      ``draft``   : [B*k_max, V] stored drafter logits (float32 or uint16 bf16 bits),
      ``target``  : [B*(k_max+1), V] stored target logits, dense by sequence
                    (row b*(k_max+1)+i is position i; i = k_max is the bonus row),
      ``drafted`` : [B, k_max] int32 drafted ids,
      ``uniforms``: [B, k_max+1] float32 (slot k_max = final-sample uniform),
      ``cfg``     : the Config.
    For a dense config the target/uniform arrays are already in the packed layout
    with k_b = k_max for every sequence.
    """
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    B, K, V = cfg.B, cfg.k_max, cfg.V
    st = np.float32 if cfg.dtype == "f32" else np.uint16
    draft = np.empty((B * K, V), dtype=st)
    target = np.empty((B * (K + 1), V), dtype=st)
    drafted = np.empty((B, K), dtype=np.int32)
    unif = np.empty((B, K + 1), dtype=np.float32)
    if cfg.kind == "c4":
        _c4_perm_cache(cfg, seed)
    if cfg.kind == "c3":
        _c3_indep_rows(cfg, seed)
    _log_rank(V)

    def do_seq(b: int) -> None:
        for i in range(K):
            r = b * K + i
            d = draft_row(cfg, seed, r)
            draft[r] = d
            drafted[b, i] = drafted_id(cfg, seed, r, d)
            target[b * (K + 1) + i] = target_row(cfg, seed, b, i, d)
        target[b * (K + 1) + K] = target_row(cfg, seed, b, K)
        unif[b] = uniform(cfg, seed, b)

    n = threads or _threads()
    if n <= 1 or B == 1:
        for b in range(B):
            do_seq(b)
    else:
        with ThreadPoolExecutor(n) as ex:
            list(ex.map(do_seq, range(B)))
    return {"draft": draft, "target": target, "drafted": drafted, "uniforms": unif, "cfg": cfg}


def pack_ragged(k: np.ndarray, k_max: int, padded_rows: np.ndarray) -> np.ndarray:
    """Host-side packing of a padded per-sequence array ``[B, k_max+1, ...]`` into
    ``[sum(k_b+1), ...]``: positions 0..k_b-1 followed by the slot-k_max entry.

    Index bookkeeping only (used by tests to build the oracle's inputs for the
    ragged workload; the device path packs with the offsets it computed).
    """
    B = len(k)
    out = []
    for b in range(B):
        kb = int(k[b])
        out.append(padded_rows[b, :kb])
        out.append(padded_rows[b, k_max:k_max + 1])
    return np.concatenate(out, axis=0)


def pack_device(padded, k, off, k_max: int):
    """Device-side packing of a padded per-sequence tensor ``[B*(k_max+1), ...]``
    (position i of sequence b at row b*(k_max+1)+i, the final slot at i = k_max) into
    the packed layout given device draft lengths ``k`` [B] and offsets ``off`` [B+1]:
    packed row off[b]+i holds position i for i < k_b and the final slot at i = k_b.
    Rows at or beyond off[B] receive arbitrary (in-bounds) copies.  Index bookkeeping
    only, with torch gather ops (no host synchronisation)."""
    import torch

    B = k.numel()
    R = B * (k_max + 1)
    p = torch.arange(R, device=padded.device, dtype=torch.int64)
    b = torch.searchsorted(off[1:].to(torch.int64).contiguous(), p, right=True).clamp_(max=B - 1)
    i = p - off.to(torch.int64)[b]
    kb = k.to(torch.int64)[b]
    src = b * (k_max + 1) + torch.where((i >= 0) & (i < kb), i, torch.full_like(i, k_max))
    return padded.index_select(0, src)
