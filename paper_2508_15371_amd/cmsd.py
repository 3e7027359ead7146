"""ctypes binding of ``libcmsd.so`` (include/cmsd.h).

Argument marshalling only: the functions below check tensor shapes/dtypes, turn
torch tensors into device pointers and the current HIP stream into a handle, and
call the C entry points of the same name.  Every step of the computation runs in
the library's HIP kernels; there is no fallback.  Importing this module raises
``ImportError`` when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcmsd.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "cmsd.h")

CMSD_OK, CMSD_ERR_ARG, CMSD_ERR_DTYPE, CMSD_ERR_LAUNCH, CMSD_ERR_SIZE = 0, 1, 2, 3, 4
CMSD_STATIC_SCRATCH_BYTES = 16 << 20     # include/cmsd.h
CMSD_F32, CMSD_BF16 = 0, 1
CMSD_MODE_STANDARD, CMSD_MODE_CM, CMSD_MODE_GREEDY = 0, 1, 2

STATS_FIELDS = ("max_logit", "sum_exp", "entropy", "margin_soft", "margin_logit", "conf", "top1", "flags")
TSTATS_FIELDS = ("max_logit", "sum_exp", "n_greater", "accept", "top1", "reserved0", "reserved1", "reserved2")


class ConfParams(C.Structure):
    _fields_ = [("lambda_ent", C.c_float), ("lambda_margin", C.c_float), ("lambda_soft", C.c_float),
                ("beta_margin", C.c_float)]


class DraftParams(C.Structure):
    _fields_ = [("k_min", C.c_int32), ("k_max", C.c_int32), ("alpha", C.c_float)]


class VerifyParams(C.Structure):
    _fields_ = [("mode", C.c_int32), ("top_beta", C.c_int32), ("tau_base", C.c_float), ("gamma", C.c_float)]


class CmsdError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: status {status} ({_lib.cmsd_status_string(status).decode()})")
        self.status = status


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2508_15371_amd.build`")
    lib = C.CDLL(LIB_PATH)
    vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
    lib.cmsd_confidence.argtypes = [vp, i32, i64, i64, i64, C.POINTER(ConfParams), vp, vp]
    lib.cmsd_confidence.restype = C.c_int
    lib.cmsd_confidence_var.argtypes = [vp, i32, i64, i64, i64, C.POINTER(ConfParams), vp, vp, vp]
    lib.cmsd_confidence_var.restype = C.c_int
    lib.cmsd_draft_len.argtypes = [vp, i32, C.POINTER(DraftParams), vp, vp, vp]
    lib.cmsd_draft_len.restype = C.c_int
    lib.cmsd_verify.argtypes = [vp, i64, vp, vp, i64, i64, vp, vp, vp, vp, i32, i32, i32, i64,
                                C.POINTER(VerifyParams), vp, vp, vp, vp, C.c_size_t, vp]
    lib.cmsd_verify_workspace_bytes.argtypes = [i32, i32, i64]
    lib.cmsd_verify_workspace_bytes.restype = C.c_size_t
    lib.cmsd_verify.restype = C.c_int
    lib.cmsd_draft_sample.argtypes = [vp, i32, i64, i64, i64, vp, vp, vp, vp, C.c_size_t, vp]
    lib.cmsd_draft_sample.restype = C.c_int
    lib.cmsd_draft_sample_workspace_bytes.argtypes = [i64, i64]
    lib.cmsd_draft_sample_workspace_bytes.restype = C.c_size_t
    lib.cmsd_logit_pass.argtypes = [vp, i64, vp, i64, vp, vp, i32, i32, i32, i64, C.POINTER(ConfParams),
                                    C.POINTER(DraftParams), C.POINTER(VerifyParams), i32, vp, vp, vp, vp, vp, vp,
                                    C.c_size_t, vp]
    lib.cmsd_logit_pass.restype = C.c_int
    lib.cmsd_set_row_events.argtypes = [C.POINTER(vp)]
    lib.cmsd_set_row_events.restype = C.c_int
    lib.cmsd_logit_pass_fused.argtypes = [vp, i64, vp, i64, vp, vp, i32, i32, i32, i64, C.POINTER(ConfParams),
                                          C.POINTER(DraftParams), C.POINTER(VerifyParams), i32, vp, vp, vp, vp, vp,
                                          vp, C.c_size_t, vp]
    lib.cmsd_logit_pass_fused.restype = C.c_int
    lib.cmsd_logit_pass_noalloc.argtypes = [vp, i64, vp, i64, vp, vp, i32, i32, i32, i64, C.POINTER(ConfParams),
                                            C.POINTER(DraftParams), C.POINTER(VerifyParams), i32, vp, vp, vp, vp,
                                            vp, vp]
    lib.cmsd_logit_pass_noalloc.restype = C.c_int
    lib.cmsd_set_row_shape.argtypes = [i32, i32]
    lib.cmsd_set_row_shape.restype = C.c_int
    lib.cmsd_set_pass_decisions.argtypes = [i32]
    lib.cmsd_set_pass_decisions.restype = C.c_int
    lib.cmsd_logit_pass_fused_workspace_bytes.argtypes = [i32, i32, i64]
    lib.cmsd_logit_pass_fused_workspace_bytes.restype = C.c_size_t
    lib.cmsd_status_string.argtypes = [C.c_int]
    lib.cmsd_status_string.restype = C.c_char_p
    lib.cmsd_version.argtypes = []
    lib.cmsd_version.restype = C.c_int32
    return lib


_lib = _load()


def lib() -> C.CDLL:
    """The loaded ``libcmsd.so`` (raw entry points, ``argtypes`` set)."""
    return _lib


def header_symbols() -> list[str]:
    """Entry points declared in include/cmsd.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:cmsd_status|const char\*|int32_t|size_t)\s+(cmsd_\w+)\s*\(", txt, re.M)))


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return CMSD_F32
    if t.dtype == torch.bfloat16:
        return CMSD_BF16
    raise TypeError(f"logits must be float32 or bfloat16, got {t.dtype}")


def _rows(t: torch.Tensor, name: str) -> tuple[int, int, int]:
    """(rows, vocab, row_stride) of a [rows, V] logit matrix with unit inner stride."""
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D [rows, vocab] tensor with unit inner stride")
    return t.shape[0], t.shape[1], t.stride(0)


def _on_device(t: torch.Tensor, name: str) -> None:
    """Checked after every size check, so those also run on host tensors."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")


def _buf(t: torch.Tensor, name: str, dtype: torch.dtype, min_elems: int, device: torch.device) -> None:
    """A caller-owned buffer: a contiguous ``dtype`` tensor on ``device`` with at
    least ``min_elems`` elements (the kernels take plain pointers and cannot check)."""
    if t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor")
    if t.numel() < min_elems:
        raise ValueError(f"{name} has {t.numel()} elements; {min_elems} are needed")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, not {t.device}")


def cmsd_set_row_shape(threads: int = 0, ring_depth: int = 0) -> None:
    """Force the row kernels' workgroup size (64/128/256) and loads-in-flight depth
    (2/3); 0 restores the per-launch choice.  Process-wide."""
    _check("cmsd_set_row_shape", _lib.cmsd_set_row_shape(int(threads), int(ring_depth)))


def cmsd_set_pass_decisions(mode: int = 0) -> None:
    """Where cmsd_logit_pass forms each sequence's decisions: 0 chosen per call, 1 a
    decision kernel's record (four launches), 2 in every final-token workgroup (three
    launches).  Bit-identical outputs.  Process-wide."""
    _check("cmsd_set_pass_decisions", _lib.cmsd_set_pass_decisions(int(mode)))


def cmsd_set_row_events(row_events) -> None:
    """Arm the next cmsd_logit_pass call of this thread to record the pair of
    recorded-once ``torch.cuda.Event`` objects just before and just after its row-pass
    launch (None disarms).  A measurement hook; results never depend on it."""
    _check("cmsd_set_row_events", _lib.cmsd_set_row_events(_events(row_events)))


def _events(evs):
    """A pair of torch.cuda.Event as the C array of two hipEvent_t, or None."""
    if evs is None:
        return None
    if len(evs) != 2 or any(e.cuda_event == 0 for e in evs):
        raise ValueError("row_events must be two torch.cuda.Event objects that have been recorded once")
    return (C.c_void_p * 2)(evs[0].cuda_event, evs[1].cuda_event)


def _check(fn: str, status: int) -> None:
    if status != CMSD_OK:
        raise CmsdError(fn, status)


def cmsd_confidence(logits: torch.Tensor, stats: torch.Tensor | None = None, *,
                    lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin: float = 1.0, stream=None) -> torch.Tensor:
    """Per-row stats of ``logits`` [rows, V] -> float32 [rows, 8] (columns STATS_FIELDS;
    ``top1`` and ``flags`` hold int32 bits: read them with ``.view(torch.int32)``)."""
    n, V, st = _rows(logits, "logits")
    if stats is None:
        stats = torch.empty((n, 8), dtype=torch.float32, device=logits.device)
    _buf(stats, "stats", torch.float32, 8 * n, logits.device)
    p = ConfParams(float(lambdas[0]), float(lambdas[1]), float(lambdas[2]), float(beta_margin))
    _on_device(logits, "logits")
    _check("cmsd_confidence", _lib.cmsd_confidence(_ptr(logits), _dtype_code(logits), n, V, st, C.byref(p),
                                                   _ptr(stats), _stream(stream)))
    return stats


def cmsd_confidence_var(logits: torch.Tensor, stats: torch.Tensor | None = None, logit_var: torch.Tensor | None = None,
                        *, lambdas=(1 / 3, 1 / 3, 1 / 3), beta_margin: float = 1.0,
                        stream=None) -> tuple[torch.Tensor, torch.Tensor]:
    """cmsd_confidence plus the variance of each row's finite logits -> (stats
    float32 [rows, 8], logit_var float32 [rows])."""
    n, V, st = _rows(logits, "logits")
    if stats is None:
        stats = torch.empty((n, 8), dtype=torch.float32, device=logits.device)
    if logit_var is None:
        logit_var = torch.empty(n, dtype=torch.float32, device=logits.device)
    _buf(stats, "stats", torch.float32, 8 * n, logits.device)
    _buf(logit_var, "logit_var", torch.float32, n, logits.device)
    p = ConfParams(float(lambdas[0]), float(lambdas[1]), float(lambdas[2]), float(beta_margin))
    _on_device(logits, "logits")
    _check("cmsd_confidence_var", _lib.cmsd_confidence_var(_ptr(logits), _dtype_code(logits), n, V, st, C.byref(p),
                                                           _ptr(stats), _ptr(logit_var), _stream(stream)))
    return stats, logit_var


def cmsd_draft_len(stats: torch.Tensor, batch: int, *, k_min: int, k_max: int, alpha: float,
                   draft_len: torch.Tensor | None = None, target_offsets: torch.Tensor | None = None,
                   stream=None) -> tuple[torch.Tensor, torch.Tensor]:
    """Draft lengths [batch] int32 and packed target offsets [batch+1] int32 from the
    drafter stats of batch*k_max rows."""
    dev = stats.device
    if draft_len is None:
        draft_len = torch.empty(batch, dtype=torch.int32, device=dev)
    if target_offsets is None:
        target_offsets = torch.empty(batch + 1, dtype=torch.int32, device=dev)
    _buf(stats, "stats", torch.float32, 8 * batch * k_max, dev)
    _buf(draft_len, "draft_len", torch.int32, batch, dev)
    _buf(target_offsets, "target_offsets", torch.int32, batch + 1, dev)
    p = DraftParams(int(k_min), int(k_max), float(alpha))
    _on_device(stats, "stats")
    _check("cmsd_draft_len", _lib.cmsd_draft_len(_ptr(stats), int(batch), C.byref(p), _ptr(draft_len),
                                                 _ptr(target_offsets), _stream(stream)))
    return draft_len, target_offsets


def cmsd_verify_workspace_bytes(batch: int, k_max: int, vocab: int) -> int:
    """Bytes of device workspace cmsd_verify needs."""
    return int(_lib.cmsd_verify_workspace_bytes(int(batch), int(k_max), int(vocab)))


def verify_workspace(batch: int, k_max: int, vocab: int, device) -> torch.Tensor:
    """A device workspace tensor for cmsd_verify (allocate once, reuse across calls)."""
    n = max(8, cmsd_verify_workspace_bytes(batch, k_max, vocab))
    return torch.empty((n + 7) // 8, dtype=torch.float64, device=device)


def cmsd_logit_pass_fused_workspace_bytes(batch: int, k_max: int, vocab: int) -> int:
    return int(_lib.cmsd_logit_pass_fused_workspace_bytes(int(batch), int(k_max), int(vocab)))


def fused_workspace(batch: int, k_max: int, vocab: int, device) -> torch.Tensor:
    """A zero-filled device workspace for cmsd_logit_pass_fused (its per-sequence
    counters must start at zero; every call leaves them zero).  Allocate once, reuse."""
    n = max(8, cmsd_logit_pass_fused_workspace_bytes(batch, k_max, vocab))
    return torch.zeros((n + 7) // 8, dtype=torch.float64, device=device)


def cmsd_verify(draft_logits: torch.Tensor, draft_stats: torch.Tensor, target_logits: torch.Tensor,
                target_offsets: torch.Tensor, draft_len: torch.Tensor, drafted: torch.Tensor,
                uniforms: torch.Tensor, *, batch: int, k_max: int, mode: int = CMSD_MODE_CM, top_beta: int = 3,
                tau_base: float = 0.1, gamma: float = 1.0, target_stats: torch.Tensor | None = None,
                n_accepted: torch.Tensor | None = None, next_token: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None, stream=None) -> tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Verification of every drafted position; returns (n_accepted [batch] int32,
    next_token [batch] int32, target_stats float32 [target_rows, 8] with int32 bits in
    columns 2..7).  ``uniforms`` may be None in GREEDY mode."""
    _, V, dst = _rows(draft_logits, "draft_logits")
    trows, V2, tst = _rows(target_logits, "target_logits")
    if V2 != V or target_logits.dtype != draft_logits.dtype:
        raise ValueError("draft and target logits must share vocab size and dtype")
    dev = target_logits.device
    if target_stats is None:
        target_stats = torch.empty((trows, 8), dtype=torch.float32, device=dev)
    if n_accepted is None:
        n_accepted = torch.empty(batch, dtype=torch.int32, device=dev)
    if next_token is None:
        next_token = torch.empty(batch, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = verify_workspace(batch, k_max, V, dev)
    drows = draft_logits.shape[0]
    if drows < batch * k_max:
        raise ValueError(f"draft_logits has {drows} rows; batch*k_max = {batch * k_max} are needed")
    if draft_logits.device != dev:
        raise ValueError("draft and target logits must be on one device")
    for name, t, dt, n in (("draft_stats", draft_stats, torch.float32, 8 * batch * k_max),
                           ("target_offsets", target_offsets, torch.int32, batch + 1),
                           ("draft_len", draft_len, torch.int32, batch),
                           ("drafted", drafted, torch.int32, batch * k_max),
                           ("uniforms", uniforms, torch.float32, trows),
                           ("target_stats", target_stats, torch.float32, 8 * trows),
                           ("n_accepted", n_accepted, torch.int32, batch),
                           ("next_token", next_token, torch.int32, batch)):
        if t is None and name == "uniforms":
            continue
        _buf(t, name, dt, n, dev)
    if workspace.dtype != torch.float64 or not workspace.is_contiguous() or workspace.device != dev:
        raise ValueError(f"workspace must be a contiguous float64 tensor on {dev}")
    p = VerifyParams(int(mode), int(top_beta), float(tau_base), float(gamma))
    _on_device(target_logits, "target_logits")
    _check("cmsd_verify", _lib.cmsd_verify(
        _ptr(draft_logits), dst, _ptr(draft_stats), _ptr(target_logits), tst, trows,
        _ptr(target_offsets), _ptr(draft_len), _ptr(drafted), _ptr(uniforms), _dtype_code(target_logits),
        int(batch), int(k_max), V, C.byref(p), _ptr(target_stats), _ptr(n_accepted), _ptr(next_token),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))
    return n_accepted, next_token, target_stats


def cmsd_draft_sample_workspace_bytes(n_rows: int, vocab: int) -> int:
    return int(_lib.cmsd_draft_sample_workspace_bytes(int(n_rows), int(vocab)))


def cmsd_draft_sample(logits: torch.Tensor, stats: torch.Tensor, uniforms: torch.Tensor,
                      drafted: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                      stream=None) -> torch.Tensor:
    """One softmax sample per row of ``logits`` [rows, V] with ``uniforms`` [rows]
    (stats from cmsd_confidence on the same logits) -> int32 [rows]."""
    n, V, st = _rows(logits, "logits")
    dev = logits.device
    if drafted is None:
        drafted = torch.empty(n, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(1, (cmsd_draft_sample_workspace_bytes(n, V) + 7) // 8), dtype=torch.float64,
                                device=dev)
    _buf(stats, "stats", torch.float32, 8 * n, dev)
    _buf(uniforms, "uniforms", torch.float32, n, dev)
    _buf(drafted, "drafted", torch.int32, n, dev)
    if workspace.dtype != torch.float64 or not workspace.is_contiguous() or workspace.device != dev:
        raise ValueError(f"workspace must be a contiguous float64 tensor on {dev}")
    _on_device(logits, "logits")
    _check("cmsd_draft_sample", _lib.cmsd_draft_sample(
        _ptr(logits), _dtype_code(logits), n, V, st, _ptr(stats), _ptr(uniforms), _ptr(drafted), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return drafted


_NO_WORKSPACE = object()     # marker: the call takes no workspace (cmsd_logit_pass_noalloc)


def _pass_args(draft_logits, target_logits, drafted, uniforms, batch, k_max, lambdas, beta_margin, k_min, alpha,
               mode, top_beta, tau_base, gamma, outs, workspace, make_workspace):
    """Checks and completes the arguments of the single-call passes."""
    drows, V, dst = _rows(draft_logits, "draft_logits")
    trows, V2, tst = _rows(target_logits, "target_logits")
    if V2 != V or target_logits.dtype != draft_logits.dtype:
        raise ValueError("draft and target logits must share vocab size and dtype")
    if drows < batch * k_max:
        raise ValueError(f"draft_logits has {drows} rows; batch*k_max = {batch * k_max} are needed")
    if trows < batch * (k_max + 1):
        raise ValueError(f"target_logits has {trows} rows; batch*(k_max+1) = {batch * (k_max + 1)} are needed")
    dev = target_logits.device
    if draft_logits.device != dev:
        raise ValueError("draft and target logits must be on one device")
    nt = batch * (k_max + 1)
    out = dict(outs)
    shapes = {"draft_stats": ((batch * k_max, 8), torch.float32), "draft_len": ((batch,), torch.int32),
              "target_stats": ((nt, 8), torch.float32), "n_accepted": ((batch,), torch.int32),
              "next_token": ((batch,), torch.int32)}
    for k, (shape, dt) in shapes.items():
        if out[k] is None:
            out[k] = torch.empty(shape, dtype=dt, device=dev)
    for name, t, dt, n in (("drafted", drafted, torch.int32, batch * k_max),
                           ("uniforms", uniforms, torch.float32, nt),
                           ("draft_stats", out["draft_stats"], torch.float32, 8 * batch * k_max),
                           ("draft_len", out["draft_len"], torch.int32, batch),
                           ("target_stats", out["target_stats"], torch.float32, 8 * nt),
                           ("n_accepted", out["n_accepted"], torch.int32, batch),
                           ("next_token", out["next_token"], torch.int32, batch)):
        if t is None and name == "uniforms":
            continue
        _buf(t, name, dt, n, dev)
    if workspace is _NO_WORKSPACE:
        pass
    elif workspace is None:
        workspace = make_workspace(batch, k_max, V, dev)
    if workspace is not _NO_WORKSPACE and (workspace.dtype != torch.float64 or not workspace.is_contiguous()
                                           or workspace.device != dev):
        raise ValueError(f"workspace must be a contiguous float64 tensor on {dev}")
    out["workspace"] = workspace
    cp = ConfParams(float(lambdas[0]), float(lambdas[1]), float(lambdas[2]), float(beta_margin))
    dp = DraftParams(int(k_min), int(k_max), float(alpha))
    vp_ = VerifyParams(int(mode), int(top_beta), float(tau_base), float(gamma))
    _on_device(target_logits, "target_logits")
    return out, dst, tst, V, cp, dp, vp_


def cmsd_logit_pass(draft_logits: torch.Tensor, target_logits: torch.Tensor, drafted: torch.Tensor,
                    uniforms: torch.Tensor | None, *, batch: int, k_max: int, lambdas=(1 / 3, 1 / 3, 1 / 3),
                    beta_margin: float = 1.0, k_min: int = 1, alpha: float = 1.0, mode: int = CMSD_MODE_CM,
                    top_beta: int = 3, tau_base: float = 0.1, gamma: float = 1.0, adaptive: bool = False,
                    draft_stats: torch.Tensor | None = None, draft_len: torch.Tensor | None = None,
                    target_stats: torch.Tensor | None = None, n_accepted: torch.Tensor | None = None,
                    next_token: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                    row_events=None, stream=None) -> dict:
    """Confidence, draft length and verification of a dense draft in one call.
    ``draft_logits`` [batch*k_max, V], ``target_logits`` [batch*(k_max+1), V] (same
    dtype), ``drafted`` int32 [batch*k_max], ``uniforms`` float32 [batch*(k_max+1)]
    (None in GREEDY mode).  ``row_events``: optional pair of recorded-once
    ``torch.cuda.Event`` objects, recorded on the call's stream just before and just
    after the row-pass launch (armed through cmsd_set_row_events right before the
    call).  Returns the output tensors by name."""
    outs = {"draft_stats": draft_stats, "draft_len": draft_len, "target_stats": target_stats,
            "n_accepted": n_accepted, "next_token": next_token}
    out, dst, tst, V, cp, dp, vp_ = _pass_args(draft_logits, target_logits, drafted, uniforms, batch, k_max, lambdas,
                                               beta_margin, k_min, alpha, mode, top_beta, tau_base, gamma, outs,
                                               workspace, verify_workspace)
    ws = out["workspace"]
    if row_events is not None:
        cmsd_set_row_events(row_events)
    _check("cmsd_logit_pass", _lib.cmsd_logit_pass(
        _ptr(draft_logits), dst, _ptr(target_logits), tst, _ptr(drafted), _ptr(uniforms),
        _dtype_code(target_logits), int(batch), int(k_max), V, C.byref(cp), C.byref(dp), C.byref(vp_),
        1 if adaptive else 0, _ptr(out["draft_stats"]), _ptr(out["draft_len"]), _ptr(out["target_stats"]),
        _ptr(out["n_accepted"]), _ptr(out["next_token"]), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return out


def cmsd_logit_pass_fused(draft_logits: torch.Tensor, target_logits: torch.Tensor, drafted: torch.Tensor,
                          uniforms: torch.Tensor | None, *, batch: int, k_max: int, lambdas=(1 / 3, 1 / 3, 1 / 3),
                          beta_margin: float = 1.0, k_min: int = 1, alpha: float = 1.0, mode: int = CMSD_MODE_CM,
                          top_beta: int = 3, tau_base: float = 0.1, gamma: float = 1.0, adaptive: bool = False,
                          draft_stats: torch.Tensor | None = None, draft_len: torch.Tensor | None = None,
                          target_stats: torch.Tensor | None = None, n_accepted: torch.Tensor | None = None,
                          next_token: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                          stream=None) -> dict:
    """cmsd_logit_pass in one launch, for small batches (a few hundred rows).  Same
    arguments and outputs; ``workspace`` must come from ``fused_workspace`` (or be
    zero-filled once before its first use) and is reused across calls."""
    outs = {"draft_stats": draft_stats, "draft_len": draft_len, "target_stats": target_stats,
            "n_accepted": n_accepted, "next_token": next_token}
    out, dst, tst, V, cp, dp, vp_ = _pass_args(draft_logits, target_logits, drafted, uniforms, batch, k_max, lambdas,
                                               beta_margin, k_min, alpha, mode, top_beta, tau_base, gamma, outs,
                                               workspace, fused_workspace)
    ws = out["workspace"]
    _check("cmsd_logit_pass_fused", _lib.cmsd_logit_pass_fused(
        _ptr(draft_logits), dst, _ptr(target_logits), tst, _ptr(drafted), _ptr(uniforms),
        _dtype_code(target_logits), int(batch), int(k_max), V, C.byref(cp), C.byref(dp), C.byref(vp_),
        1 if adaptive else 0, _ptr(out["draft_stats"]), _ptr(out["draft_len"]), _ptr(out["target_stats"]),
        _ptr(out["n_accepted"]), _ptr(out["next_token"]), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return out


def cmsd_logit_pass_noalloc(draft_logits: torch.Tensor, target_logits: torch.Tensor, drafted: torch.Tensor,
                            uniforms: torch.Tensor | None, *, batch: int, k_max: int, lambdas=(1 / 3, 1 / 3, 1 / 3),
                            beta_margin: float = 1.0, k_min: int = 1, alpha: float = 1.0, mode: int = CMSD_MODE_CM,
                            top_beta: int = 3, tau_base: float = 0.1, gamma: float = 1.0, adaptive: bool = False,
                            draft_stats: torch.Tensor | None = None, draft_len: torch.Tensor | None = None,
                            target_stats: torch.Tensor | None = None, n_accepted: torch.Tensor | None = None,
                            next_token: torch.Tensor | None = None, stream=None) -> dict:
    """cmsd_logit_pass on the library's static scratch instead of a workspace (the
    call allocates no device memory; pass preallocated outputs to allocate nothing
    here either).  Same arguments and outputs, without ``workspace``/``row_events``."""
    outs = {"draft_stats": draft_stats, "draft_len": draft_len, "target_stats": target_stats,
            "n_accepted": n_accepted, "next_token": next_token}
    out, dst, tst, V, cp, dp, vp_ = _pass_args(draft_logits, target_logits, drafted, uniforms, batch, k_max, lambdas,
                                               beta_margin, k_min, alpha, mode, top_beta, tau_base, gamma, outs,
                                               _NO_WORKSPACE, None)
    del out["workspace"]
    _check("cmsd_logit_pass_noalloc", _lib.cmsd_logit_pass_noalloc(
        _ptr(draft_logits), dst, _ptr(target_logits), tst, _ptr(drafted), _ptr(uniforms),
        _dtype_code(target_logits), int(batch), int(k_max), V, C.byref(cp), C.byref(dp), C.byref(vp_),
        1 if adaptive else 0, _ptr(out["draft_stats"]), _ptr(out["draft_len"]), _ptr(out["target_stats"]),
        _ptr(out["n_accepted"]), _ptr(out["next_token"]), _stream(stream)))
    return out
