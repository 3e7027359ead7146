"""The C ABI on the host: the library loads, exports every declared entry point, and
rejects invalid arguments before enqueuing anything (no GPU needed: these calls
return before any HIP call)."""
import ctypes as C

import pytest

cm = pytest.importorskip("paper_2508_15371_amd.cmsd")

P = 0x10000          # fake, aligned device addresses: never dereferenced on these paths


def test_exports_every_declared_symbol():
    syms = cm.header_symbols()
    assert set(syms) >= {"cmsd_confidence", "cmsd_confidence_var", "cmsd_draft_len", "cmsd_verify",
                         "cmsd_verify_workspace_bytes",
                         "cmsd_draft_sample", "cmsd_draft_sample_workspace_bytes", "cmsd_status_string",
                         "cmsd_version", "cmsd_logit_pass", "cmsd_logit_pass_fused",
                         "cmsd_logit_pass_fused_workspace_bytes", "cmsd_logit_pass_noalloc",
                         "cmsd_set_row_shape", "cmsd_set_pass_decisions", "cmsd_set_row_events"}
    lib = cm.lib()
    for s in syms:
        assert hasattr(lib, s), s
    assert lib.cmsd_version() == (1 << 16) | 7
    assert lib.cmsd_status_string(0) == b"ok"
    assert lib.cmsd_status_string(1) == b"invalid argument"
    assert lib.cmsd_status_string(4) == b"problem larger than the static scratch"


def test_header_constants_match_binding():
    import re
    txt = open(cm.HEADER).read()
    assert re.search(r"#define CMSD_STATIC_SCRATCH_BYTES \(16u << 20\)", txt)
    assert cm.CMSD_STATIC_SCRATCH_BYTES == 16 << 20
    assert re.search(r"CMSD_ERR_SIZE = 4", txt) and cm.CMSD_ERR_SIZE == 4


@pytest.mark.parametrize("threads,depth,want", [
    (0, 0, cm.CMSD_OK), (64, 2, cm.CMSD_OK), (128, 3, cm.CMSD_OK), (256, 0, cm.CMSD_OK),
    (32, 0, cm.CMSD_ERR_ARG), (512, 0, cm.CMSD_ERR_ARG), (-64, 0, cm.CMSD_ERR_ARG),
    (0, 1, cm.CMSD_ERR_ARG), (0, 4, cm.CMSD_ERR_ARG), (64, -2, cm.CMSD_ERR_ARG),
])
def test_set_row_shape(threads, depth, want):
    lib = cm.lib()
    try:
        assert lib.cmsd_set_row_shape(threads, depth) == want
    finally:
        assert lib.cmsd_set_row_shape(0, 0) == cm.CMSD_OK


@pytest.mark.parametrize("mode,want", [(0, cm.CMSD_OK), (1, cm.CMSD_OK), (2, cm.CMSD_OK),
                                       (-1, cm.CMSD_ERR_ARG), (3, cm.CMSD_ERR_ARG)])
def test_set_pass_decisions(mode, want):
    lib = cm.lib()
    try:
        assert lib.cmsd_set_pass_decisions(mode) == want
    finally:
        assert lib.cmsd_set_pass_decisions(0) == cm.CMSD_OK


def test_set_row_events():
    # arming and disarming touch no device: a pair with a null entry is refused, and a
    # rejected cmsd_logit_pass call disarms what was armed (fake handles, never used)
    lib = cm.lib()
    assert lib.cmsd_set_row_events((C.c_void_p * 2)(P, None)) == cm.CMSD_ERR_ARG
    assert lib.cmsd_set_row_events(None) == cm.CMSD_OK
    assert lib.cmsd_set_row_events((C.c_void_p * 2)(P, P + 64)) == cm.CMSD_OK
    assert _lpass(dtype=3) == cm.CMSD_ERR_DTYPE
    assert lib.cmsd_set_row_events(None) == cm.CMSD_OK


def _conf(**kw):
    a = dict(logits=P, dtype=cm.CMSD_BF16, n=4, V=1024, stride=1024, p=cm.ConfParams(0.25, 0.25, 0.5, 1.0), out=P)
    a.update(kw)
    return cm.lib().cmsd_confidence(a["logits"], a["dtype"], a["n"], a["V"], a["stride"],
                                    C.byref(a["p"]) if a["p"] is not None else None, a["out"], None)


@pytest.mark.parametrize("kw,want", [
    (dict(dtype=5), cm.CMSD_ERR_DTYPE),
    (dict(p=None), cm.CMSD_ERR_ARG),
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(stride=1000), cm.CMSD_ERR_ARG),
    (dict(n=-1), cm.CMSD_ERR_ARG),
    (dict(logits=None), cm.CMSD_ERR_ARG),
    (dict(out=None), cm.CMSD_ERR_ARG),
    (dict(logits=P + 1), cm.CMSD_ERR_ARG),                       # misaligned bf16 pointer
    (dict(p=cm.ConfParams(0.5, 0.5, 0.5, 1.0)), cm.CMSD_ERR_ARG),  # weights do not sum to 1
    (dict(p=cm.ConfParams(-0.1, 0.6, 0.5, 1.0)), cm.CMSD_ERR_ARG),
    (dict(p=cm.ConfParams(0.25, 0.25, 0.5, 0.0)), cm.CMSD_ERR_ARG),  # beta_margin must be > 0
    (dict(p=cm.ConfParams(0.25, 0.25, 0.5, float("inf"))), cm.CMSD_ERR_ARG),
    (dict(n=0, logits=None, out=None), cm.CMSD_OK),             # empty input: nothing enqueued
])
def test_confidence_argument_errors(kw, want):
    assert _conf(**kw) == want


@pytest.mark.parametrize("k_min,k_max,alpha,batch,want", [
    (0, 8, 1.0, 4, cm.CMSD_ERR_ARG),
    (9, 8, 1.0, 4, cm.CMSD_ERR_ARG),
    (1, 5000, 1.0, 4, cm.CMSD_ERR_ARG),
    (1, 8, 0.0, 4, cm.CMSD_ERR_ARG),
    (1, 8, 1.5, 4, cm.CMSD_ERR_ARG),
    (1, 8, float("nan"), 4, cm.CMSD_ERR_ARG),
    (1, 8, 1.0, -1, cm.CMSD_ERR_ARG),
])
def test_draft_len_argument_errors(k_min, k_max, alpha, batch, want):
    p = cm.DraftParams(k_min, k_max, alpha)
    assert cm.lib().cmsd_draft_len(P, batch, C.byref(p), P, P, None) == want


def _verify(**kw):
    a = dict(dl=P, ds=1024, dst=P, tl=P, ts=1024, trows=90, off=P, k=P, dr=P, u=P, dtype=cm.CMSD_BF16,
             B=10, K=8, V=1024, p=cm.VerifyParams(1, 3, 0.1, 1.0), tst=P, na=P, nt=P, ws=P, wsb=1 << 20)
    a.update(kw)
    return cm.lib().cmsd_verify(a["dl"], a["ds"], a["dst"], a["tl"], a["ts"], a["trows"], a["off"], a["k"],
                                a["dr"], a["u"], a["dtype"], a["B"], a["K"], a["V"],
                                C.byref(a["p"]) if a["p"] is not None else None, a["tst"], a["na"], a["nt"],
                                a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,want", [
    (dict(dtype=9), cm.CMSD_ERR_DTYPE),
    (dict(p=None), cm.CMSD_ERR_ARG),
    (dict(p=cm.VerifyParams(3, 3, 0.1, 1.0)), cm.CMSD_ERR_ARG),
    (dict(p=cm.VerifyParams(1, -1, 0.1, 1.0)), cm.CMSD_ERR_ARG),
    (dict(p=cm.VerifyParams(1, 3, float("inf"), 1.0)), cm.CMSD_ERR_ARG),
    (dict(p=cm.VerifyParams(1, 3, 0.1, float("nan"))), cm.CMSD_ERR_ARG),
    (dict(K=0), cm.CMSD_ERR_ARG),
    (dict(K=5000), cm.CMSD_ERR_ARG),
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(ds=1000), cm.CMSD_ERR_ARG),
    (dict(ts=1000), cm.CMSD_ERR_ARG),
    (dict(trows=0), cm.CMSD_ERR_ARG),
    (dict(B=-2), cm.CMSD_ERR_ARG),
    (dict(u=None), cm.CMSD_ERR_ARG),
    (dict(na=None), cm.CMSD_ERR_ARG),
    (dict(tl=P + 1), cm.CMSD_ERR_ARG),
    (dict(dr=P + 2), cm.CMSD_ERR_ARG),
    (dict(ws=None), cm.CMSD_ERR_ARG),
    (dict(wsb=16), cm.CMSD_ERR_ARG),                              # workspace too small
    (dict(ws=P + 4), cm.CMSD_ERR_ARG),                            # misaligned workspace
    (dict(B=0, dl=None, tl=None, ws=None, wsb=0), cm.CMSD_OK),
    # launches past 2^32 work-items (the workspace and rows are ample, so only the launch
    # sizes reject): 2^23 * 9 (sequence, position) groups of 64 threads, 2^24 sampling
    # groups of 256, 2^20 sequences * 129 slices at V = 2^17
    (dict(B=1 << 23, K=8, trows=1 << 30, wsb=1 << 62), cm.CMSD_ERR_ARG),
    (dict(B=1 << 24, K=1, trows=1 << 30, wsb=1 << 62), cm.CMSD_ERR_ARG),
    (dict(B=1 << 20, K=1, V=1 << 17, ds=1 << 17, ts=1 << 17, trows=1 << 30, wsb=1 << 62), cm.CMSD_ERR_ARG),
])

def test_verify_argument_errors(kw, want):
    assert _verify(**kw) == want


def test_workspace_size():
    f = cm.lib().cmsd_verify_workspace_bytes
    assert f(0, 8, 1000) == 0 and f(4, 8, 1) == 0 and f(4, 0, 1000) == 0 and f(4, 5000, 1000) == 0
    # per sequence: one 32-byte record per slice of 256 16-byte units (+ head and
    # tail) and one 32-byte record per target row position
    assert f(256, 16, 128256) == 256 * (32 * (((128256 // 4 + 2) + 255) // 256) + 17 * 32)
    assert f(1, 1, 2) == 32 + 2 * 32


@pytest.mark.parametrize("kw,want", [
    (dict(dtype=4), cm.CMSD_ERR_DTYPE),
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(stride=10), cm.CMSD_ERR_ARG),
    (dict(u=None), cm.CMSD_ERR_ARG),
    (dict(ws=None), cm.CMSD_ERR_ARG),
    (dict(wsb=8), cm.CMSD_ERR_ARG),
    (dict(logits=P + 1), cm.CMSD_ERR_ARG),
    (dict(n=0, logits=None, ws=None, wsb=0), cm.CMSD_OK),
    (dict(n=1 << 24, wsb=1 << 62), cm.CMSD_ERR_ARG),             # 2^24 sampling groups of 256 threads
    (dict(n=1 << 22, V=1 << 17, stride=1 << 17, wsb=1 << 62), cm.CMSD_ERR_ARG),  # 2^22 rows * 129 slices
])
def test_draft_sample_argument_errors(kw, want):
    a = dict(logits=P, dtype=cm.CMSD_BF16, n=8, V=1000, stride=1000, st=P, u=P, out=P, ws=P, wsb=1 << 20)
    a.update(kw)
    assert cm.lib().cmsd_draft_sample(a["logits"], a["dtype"], a["n"], a["V"], a["stride"], a["st"], a["u"],
                                      a["out"], a["ws"], a["wsb"], None) == want
    f = cm.lib().cmsd_draft_sample_workspace_bytes
    assert f(0, 100) == 0 and f(3, 1) == 0 and f(3, 4096) == 3 * 32 * ((4096 // 4 + 2 + 255) // 256)


def _lpass(**kw):
    a = dict(dl=P, ds=1024, tl=P, ts=1024, dr=P, u=P, dtype=cm.CMSD_BF16, B=4, K=8, V=1024,
             cp=cm.ConfParams(0.25, 0.25, 0.5, 1.0), dp=cm.DraftParams(1, 8, 1.0), vp=cm.VerifyParams(1, 3, 0.1, 1.0),
             ad=0, dst=P, kl=P, tst=P, na=P, nt=P, ws=P, wsb=1 << 20)
    a.update(kw)
    ref = lambda x: C.byref(x) if x is not None else None  # noqa: E731
    return cm.lib().cmsd_logit_pass(a["dl"], a["ds"], a["tl"], a["ts"], a["dr"], a["u"], a["dtype"], a["B"], a["K"],
                                    a["V"], ref(a["cp"]), ref(a["dp"]), ref(a["vp"]), a["ad"], a["dst"], a["kl"],
                                    a["tst"], a["na"], a["nt"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,want", [
    (dict(dtype=3), cm.CMSD_ERR_DTYPE),
    (dict(cp=None), cm.CMSD_ERR_ARG),
    (dict(dp=None), cm.CMSD_ERR_ARG),
    (dict(vp=None), cm.CMSD_ERR_ARG),
    (dict(cp=cm.ConfParams(0.5, 0.5, 0.5, 1.0)), cm.CMSD_ERR_ARG),
    (dict(dp=cm.DraftParams(1, 7, 1.0)), cm.CMSD_ERR_ARG),          # draft k_max differs from k_max
    (dict(dp=cm.DraftParams(9, 8, 1.0)), cm.CMSD_ERR_ARG),
    (dict(dp=cm.DraftParams(1, 8, 0.0)), cm.CMSD_ERR_ARG),
    (dict(vp=cm.VerifyParams(7, 3, 0.1, 1.0)), cm.CMSD_ERR_ARG),
    (dict(K=0, dp=cm.DraftParams(1, 0, 1.0)), cm.CMSD_ERR_ARG),
    (dict(K=64, dp=cm.DraftParams(1, 64, 1.0)), cm.CMSD_ERR_ARG),   # at most 63 drafts per sequence
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(ws=None), cm.CMSD_ERR_ARG),
    (dict(wsb=64), cm.CMSD_ERR_ARG),                                # workspace too small
    (dict(ws=P + 4), cm.CMSD_ERR_ARG),
    (dict(ds=1000), cm.CMSD_ERR_ARG),
    (dict(ts=1000), cm.CMSD_ERR_ARG),
    (dict(ad=2), cm.CMSD_ERR_ARG),
    (dict(B=-1), cm.CMSD_ERR_ARG),
    (dict(u=None), cm.CMSD_ERR_ARG),                                # needed outside GREEDY mode
    (dict(dr=None), cm.CMSD_ERR_ARG),
    (dict(kl=None), cm.CMSD_ERR_ARG),
    (dict(tl=P + 1), cm.CMSD_ERR_ARG),
    (dict(na=P + 2), cm.CMSD_ERR_ARG),
    (dict(B=0, dl=None, tl=None, dr=None, ws=None, wsb=0), cm.CMSD_OK),
    # launches past 2^32 work-items: 2^23 * 9 rows of 64 threads, 2^24 sampling groups,
    # 2^20 sequences * 129 slices at V = 2^17
    (dict(B=1 << 23, K=4, dp=cm.DraftParams(1, 4, 1.0), wsb=1 << 62), cm.CMSD_ERR_ARG),
    (dict(B=1 << 24, K=1, dp=cm.DraftParams(1, 1, 1.0), wsb=1 << 62), cm.CMSD_ERR_ARG),
    (dict(B=1 << 20, K=1, V=1 << 17, ds=1 << 17, ts=1 << 17, dp=cm.DraftParams(1, 1, 1.0), wsb=1 << 62),
     cm.CMSD_ERR_ARG),
])
def test_logit_pass_argument_errors(kw, want):
    assert _lpass(**kw) == want


def _fpass(**kw):
    a = dict(dl=P, ds=1024, tl=P, ts=1024, dr=P, u=P, dtype=cm.CMSD_BF16, B=4, K=8, V=1024,
             cp=cm.ConfParams(0.25, 0.25, 0.5, 1.0), dp=cm.DraftParams(1, 8, 1.0), vp=cm.VerifyParams(1, 3, 0.1, 1.0),
             ad=0, dst=P, kl=P, tst=P, na=P, nt=P, ws=P, wsb=1 << 20)
    a.update(kw)
    ref = lambda x: C.byref(x) if x is not None else None  # noqa: E731
    return cm.lib().cmsd_logit_pass_fused(a["dl"], a["ds"], a["tl"], a["ts"], a["dr"], a["u"], a["dtype"], a["B"],
                                          a["K"], a["V"], ref(a["cp"]), ref(a["dp"]), ref(a["vp"]), a["ad"], a["dst"],
                                          a["kl"], a["tst"], a["na"], a["nt"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,want", [
    (dict(dtype=3), cm.CMSD_ERR_DTYPE),
    (dict(cp=None), cm.CMSD_ERR_ARG),
    (dict(dp=cm.DraftParams(1, 7, 1.0)), cm.CMSD_ERR_ARG),
    (dict(K=64, dp=cm.DraftParams(1, 64, 1.0)), cm.CMSD_ERR_ARG),
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(ws=None), cm.CMSD_ERR_ARG),
    (dict(ws=P + 4), cm.CMSD_ERR_ARG),
    (dict(u=None), cm.CMSD_ERR_ARG),
    (dict(nt=None), cm.CMSD_ERR_ARG),
    (dict(B=-1), cm.CMSD_ERR_ARG),
    (dict(B=0, dl=None, tl=None, dr=None, ws=None, wsb=0), cm.CMSD_OK),
    (dict(B=1 << 22, K=2, dp=cm.DraftParams(1, 2, 1.0), wsb=1 << 62), cm.CMSD_ERR_ARG),  # 5 * 2^22 rows of 256
])
def test_logit_pass_fused_argument_errors(kw, want):
    assert _fpass(**kw) == want


def test_logit_pass_fused_workspace():
    f = cm.lib().cmsd_logit_pass_fused_workspace_bytes
    v = cm.lib().cmsd_verify_workspace_bytes
    # the verify workspace, then one 4-byte counter per sequence (rounded up to 8 bytes)
    assert f(8, 8, 32000) == v(8, 8, 32000) + 32
    assert f(3, 8, 32000) == v(3, 8, 32000) + 16
    assert f(0, 8, 32000) == 0 and f(4, 64, 32000) == 0 and f(4, 8, 1) == 0
    # exactly the verify workspace is one counter area too small
    assert _fpass(wsb=v(4, 8, 1024)) == cm.CMSD_ERR_ARG
    assert _fpass(wsb=f(4, 8, 1024) - 1) == cm.CMSD_ERR_ARG


def _npass(**kw):
    a = dict(dl=P, ds=1024, tl=P, ts=1024, dr=P, u=P, dtype=cm.CMSD_BF16, B=4, K=8, V=1024,
             cp=cm.ConfParams(0.25, 0.25, 0.5, 1.0), dp=cm.DraftParams(1, 8, 1.0), vp=cm.VerifyParams(1, 3, 0.1, 1.0),
             ad=0, dst=P, kl=P, tst=P, na=P, nt=P)
    a.update(kw)
    ref = lambda x: C.byref(x) if x is not None else None  # noqa: E731
    return cm.lib().cmsd_logit_pass_noalloc(a["dl"], a["ds"], a["tl"], a["ts"], a["dr"], a["u"], a["dtype"], a["B"],
                                            a["K"], a["V"], ref(a["cp"]), ref(a["dp"]), ref(a["vp"]), a["ad"],
                                            a["dst"], a["kl"], a["tst"], a["na"], a["nt"], None)


# every case returns before any HIP call (argument checks, then the scratch bound)
@pytest.mark.parametrize("kw,want", [
    (dict(dtype=3), cm.CMSD_ERR_DTYPE),
    (dict(cp=None), cm.CMSD_ERR_ARG),
    (dict(dp=cm.DraftParams(1, 7, 1.0)), cm.CMSD_ERR_ARG),
    (dict(K=64, dp=cm.DraftParams(1, 64, 1.0)), cm.CMSD_ERR_ARG),
    (dict(V=1), cm.CMSD_ERR_ARG),
    (dict(u=None), cm.CMSD_ERR_ARG),
    (dict(nt=None), cm.CMSD_ERR_ARG),
    (dict(tl=P + 1), cm.CMSD_ERR_ARG),
    (dict(ad=2), cm.CMSD_ERR_ARG),
    (dict(B=-1), cm.CMSD_ERR_ARG),
    (dict(B=0, dl=None, tl=None, dr=None), cm.CMSD_OK),
    # larger than the 16 MiB static scratch: rejected, nothing enqueued
    (dict(B=4096, K=16, V=128256, ds=128256, ts=128256, dp=cm.DraftParams(1, 16, 1.0)), cm.CMSD_ERR_SIZE),
    (dict(B=1, K=1, V=2**31 - 1, ds=2**31 - 1, ts=2**31 - 1, dp=cm.DraftParams(1, 1, 1.0)), cm.CMSD_ERR_SIZE),
])
def test_logit_pass_noalloc_argument_errors(kw, want):
    assert _npass(**kw) == want


def test_noalloc_scratch_bound_is_the_verify_workspace():
    # the bound is exactly cmsd_verify_workspace_bytes <= CMSD_STATIC_SCRATCH_BYTES:
    # per sequence at V = 128256, k_max = 16: 126 slice records + 17 row slots of 32 B
    v = cm.lib().cmsd_verify_workspace_bytes
    per = v(1, 16, 128256)
    assert per == 32 * (126 + 17)
    fit = (16 << 20) // per
    assert v(fit, 16, 128256) <= 16 << 20 < v(fit + 1, 16, 128256)
    big = dict(K=16, V=128256, ds=128256, ts=128256, dp=cm.DraftParams(1, 16, 1.0))
    assert _npass(B=fit + 1, **big) == cm.CMSD_ERR_SIZE
