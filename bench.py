"""Benchmark of the logit pass (confidence + draft length + verify) on one MI355X.

One step = one decoding iteration of the hot path over a resident synthetic batch:
drafter stats over all drafter rows, the draft lengths, and verification of all target
rows (accept decisions, prefix scan, final residual/bonus sample).  On the dense
workloads a step is one cmsd_logit_pass call (a joint row pass over drafter and target
rows, then the final-token pass); on the ragged one, whose target rows are packed by
the draft lengths, it is cmsd_confidence + cmsd_draft_len + cmsd_verify (--path calls
forces the separate calls everywhere).  Prints one JSON line.  Default workload: B=256
sequences, k_max=16, V=128256, bf16 (the largest configuration; inputs 2.17 GB).

Inputs are resident in HBM before timing; workloads smaller than 512 MiB rotate copies of
their logits between steps (``--no-rotate`` reuses one).  HIP events around the roofline
kernel in the middle step of every 64 timed steps give its achieved bandwidth (denser event markers slow
the host-bound one-sequence steps: b1 at one step in 16 went from 23 to 100 us per step
in some runs); after the timed region the
bench times each of the three calls separately, then a bare read of the roofline
kernel's rows in its grid shape (``read_ceiling``: what one launch of those bytes can
reach) and, with ``--extras``, the drafting sampler and the logit-variance pass; the CPU
oracle runs last on the host.

``--streams G`` splits the batch into G sequence groups, each with its own calls on its
own stream, so one group's final-token kernels (latency-bound) overlap another group's
row pass.  The roofline kernel is then group 0's launch, timed while the other groups'
kernels share the chip: its bytes are one group's, and its rate is what it reaches
beside them, not alone (no read ceiling or counter traffic is reported then).  With one
group (the default), the bench also times the same steps over ``--overlap`` groups (2)
after the timed region and reports their throughput under ``overlap``.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4|c5|c5m|c3|c2|v152k|tiny|b1]
                  [--mode cm|standard] [--path auto|pass|fused|calls] [--streams G] [--overlap G]
                  [--event-every N]
                  [--capacity-rows] [--no-rotate] [--extras] [--no-read-ceiling] [--no-cpu-baseline]
                  [--row-shape THREADS,DEPTH] [--copy-probe MIB]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0   # MI355X HBM3E

# HBM bytes per launch of each workload's roofline kernel, from two rocprofv3 --pmc
# runs (FETCH_SIZE, WRITE_SIZE) scaled by what the same counters read for a 1 GiB
# device copy (x2.0 and x1.0).  Valid only for the kernel code they were taken on
# (kernel_code_hash(): sha256 prefix of the .hip file's code without comments);
# otherwise "traffic" is reported null.
TRAFFIC = {"kernel_code_sha256_16": "9caa4009932a4e5a",
           "k_row_pass_c4": 2170.51e6 + 0.270e6, "k_confidence_c4": 1052.88e6 + 0.131e6,
           "k_confidence_c5": 524.71e6 + 0.262e6, "k_confidence_c5m": 524.70e6 + 0.262e6,
           "k_row_pass_c3": 112.82e6 + 0.035e6, "k_row_pass_c2": 9.15e6 + 0.004e6,
           "k_row_pass_v152k": 331.52e6 + 0.035e6,
           "k_row_pass_c4f": 4340.33e6 + 0.270e6,
           "profile": "profiles/<workload>_cm_logit_pass.md"}


def _cpu_baseline_worker(args):
    """Time the CPU oracle on one sequence of the workload (generation untimed)."""
    name, seed, b, mode = args
    import workloads as W
    from oracle import cmsd_oracle as O
    cfg = W.CONFIGS[name]
    K, V = cfg.k_max, cfg.V
    zd_s = [W.draft_row(cfg, seed, b * K + i) for i in range(K)]
    zt_s = [W.target_row(cfg, seed, b, i, zd_s[i]) for i in range(K)] + [W.target_row(cfg, seed, b, K)]
    drafted = [W.drafted_id(cfg, seed, b * K + i, zd_s[i]) for i in range(K)]
    unif = W.uniform(cfg, seed, b)
    t0 = time.perf_counter()
    zd = [O.decode_logits(z, cfg.dtype) for z in zd_s]
    zt = [O.decode_logits(z, cfg.dtype) for z in zt_s]
    lam = (1 / 3, 1 / 3, 1 / 3)
    C = np.array([[O.confidence(O.row_stats(z), V, lam, 1.0) for z in zd]])
    k_b = int(O.draft_len(C, 1, K, 1.0)[0][0]) if cfg.ragged else K
    # ragged: the verifier scored positions 0..k_b-1 and the final slot
    zt_b = zt[:k_b] + [zt[K]]
    u_b = np.concatenate([unif[:k_b], unif[K:]])
    O.verify_sequence(zt_b, zd, drafted, u_b, C[0], k_b, mode, 3, float(np.float32(0.1)), 1.0)
    return K + k_b + 1, time.perf_counter() - t0


def cpu_baseline(name: str, seed: int, mode: int, budget_s: float = 20.0) -> dict:
    """Oracle rows/s on the host cores over a bounded sample of sequences."""
    from concurrent.futures import ProcessPoolExecutor
    import workloads as W
    cfg = W.CONFIGS[name]
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:
        ncpu = os.cpu_count() or 1
    # one process per host core this process may run on, at most 16 (one GPU's
    # share of its host); the line states both the cores used and the host's count
    workers = max(1, min(16, ncpu))
    # estimate the per-sequence cost with one sequence, then size the sample to the budget
    rows1, t1 = _cpu_baseline_worker((name, seed, 0, mode))
    per_worker = max(1, int(budget_s / max(t1, 1e-3)) // 2)
    nseq = min(cfg.B, workers * per_worker)
    with ProcessPoolExecutor(workers) as ex:
        res = list(ex.map(_cpu_baseline_worker, [(name, seed, b, mode) for b in range(nseq)]))
    # workers run concurrently: aggregate rate = sum over workers of (rows / oracle time)
    by_worker = np.array_split(np.arange(nseq), workers)
    rate = 0.0
    for idx in by_worker:
        if len(idx):
            rate += sum(res[i][0] for i in idx) / sum(res[i][1] for i in idx)
    return {"value": rate, "unit": "rows/s", "cores": workers, "kind": "oracle",
            "host_cpus": ncpu, "host_cpus_online": os.cpu_count(), "cpu_model": _cpu_model(),
            "core_cap": f"min(16, {ncpu} cores available to the process)",
            "sample": f"{nseq} of {cfg.B} sequences of {name} (each {cfg.k_max} drafter + "
                      f"{'k_b+1' if cfg.ragged else cfg.k_max + 1} target rows, V={cfg.V}), numpy fp64, "
                      f"{workers} processes"}


def _cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or the platform's processor string."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def kernel_code_hash() -> str:
    """sha256 prefix of the kernel source's code: comments and blank space are
    dropped first, so an edit to comments alone keeps the measured traffic valid."""
    import hashlib
    import re
    src = open(os.path.join(ROOT, "paper_2508_15371_amd", "csrc", "cmsd.hip")).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    code = " ".join(src.split())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def _traffic(kernel: str, workload: str):
    """Measured HBM bytes per launch of `kernel`, if the kernel code is the profiled one."""
    key = f"{kernel}_{workload}"
    if kernel_code_hash() != TRAFFIC["kernel_code_sha256_16"] or key not in TRAFFIC:
        return None
    return TRAFFIC[key]


def extras(cmsd, groups, sets, n_sets, stream, cfg, steps) -> dict:
    """Per-call time of the calls around the step that it does not run: the drafting
    sampler (an exact softmax sample per drafter row, from the row stats) and the
    confidence pass with the logit-variance moment, each over all drafter rows."""
    import torch
    dev = torch.device("cuda:0")
    n = max(3, steps // 4)
    out = {}
    for name in ("cmsd_draft_sample", "cmsd_confidence_var"):
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]
        for i, e in enumerate(ev):
            for gi, (lpg, _, _) in enumerate(groups):
                draft = sets[gi][i % n_sets][0]
                rows = draft.shape[0]
                if name == "cmsd_draft_sample":
                    if not hasattr(lpg, "_xs"):
                        ws = torch.empty((cmsd.cmsd_draft_sample_workspace_bytes(rows, cfg.V) + 7) // 8,
                                         dtype=torch.float64, device=dev)
                        lpg._xs = (torch.rand(rows, device=dev), torch.empty(rows, dtype=torch.int32, device=dev), ws)
                    u, drafted, ws = lpg._xs
                    if gi == 0:
                        e[0].record(stream)
                    cmsd.cmsd_draft_sample(draft, lpg.stats, u, drafted=drafted, workspace=ws, stream=stream)
                else:
                    if not hasattr(lpg, "_xv"):
                        lpg._xv = torch.empty(rows, dtype=torch.float32, device=dev)
                    if gi == 0:
                        e[0].record(stream)
                    cmsd.cmsd_confidence_var(draft, lpg.stats, lpg._xv, stream=stream)
            e[1].record(stream)
        torch.cuda.synchronize()
        t = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e-3
        nbytes = cfg.draft_rows * cfg.V * cfg.elem_bytes
        out[name] = {"ms": t * 1e3, "logit_gbps": nbytes / t / 1e9, "rows": cfg.draft_rows}
    return out


def read_ceiling(sets, n_sets, cfg, R_t, use_pass, stream, steps, t_roof) -> dict:
    """Bare-read ceiling of the roofline kernel's launch: the same rows (drafter rows,
    then the target rows on the joint pass), the same one-workgroup-per-row grid and
    the same nontemporal 16-byte loads, nothing reduced, timed with HIP events around
    each launch like the roofline kernel.  Reports every workgroup size / loads-in-flight
    shape and the roofline kernel's time over the fastest bare read."""
    import ctypes as C
    import torch
    from paper_2508_15371_amd import build as B
    if not os.path.exists(B.PROBE_LIB):
        return {"error": f"{B.PROBE_LIB} is not built"}
    lib = C.CDLL(B.PROBE_LIB)
    i64, vp = C.c_int64, C.c_void_p
    lib.cmsd_probe_read_rows.argtypes = [vp, i64, i64, vp, i64, i64, i64, C.c_int, C.c_int, vp, vp]
    lib.cmsd_probe_read_rows.restype = C.c_int
    sink = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    s = cfg.elem_bytes
    row_bytes = cfg.V * s
    rows_b = R_t if use_pass else 0
    n = max(20, steps // 4)

    def launch(i, bd, unroll):
        a = sets[0][i % n_sets]
        draft, target = a[0], a[1]
        rc = lib.cmsd_probe_read_rows(draft.data_ptr(), draft.shape[0], draft.stride(0) * s,
                                      target.data_ptr(), rows_b, target.stride(0) * s, row_bytes,
                                      bd, unroll, sink.data_ptr(), stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"cmsd_probe_read_rows: status {rc}")

    shapes = {}
    nbytes = (cfg.draft_rows + rows_b) * row_bytes
    for bd in (64, 128, 256):
        for unroll in (4, 8):
            for i in range(10):
                launch(i, bd, unroll)
            ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]
            for i, e in enumerate(ev):
                e[0].record(stream)
                launch(i, bd, unroll)
                e[1].record(stream)
            torch.cuda.synchronize()
            t = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e-3
            shapes[f"bd{bd}_u{unroll}"] = {"us": t * 1e6, "gbps": nbytes / t / 1e9}
    best = min(shapes, key=lambda k: shapes[k]["us"])
    return {"kernel": "k_read_rows", "bytes": nbytes, "launches": n, "by_shape": shapes, "best": best,
            "best_gbps": shapes[best]["gbps"], "roofline_kernel_time_over_read": t_roof / (shapes[best]["us"] * 1e-6)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the chip's clocks settle over the first ~100 steps of this load (steps 1-50 run
    # ~3 % slower), so the default warms up for 100 steps and times 500 (~0.2 s on the default workload)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="c4", choices=["tiny", "b1", "c2", "c3", "c4", "c4f", "c5", "c5m", "v152k"])
    ap.add_argument("--mode", default="cm", choices=["cm", "standard"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--path", default="auto", choices=["auto", "pass", "fused", "calls"],
                    help="one cmsd_logit_pass call per step (dense layouts; auto: dense workloads), one "
                         "cmsd_logit_pass_fused call (one launch, for small batches), or the three separate calls")
    ap.add_argument("--streams", type=int, default=1, metavar="G",
                    help="split the batch into G sequence groups, each on its own stream (not with --path fused)")
    ap.add_argument("--overlap", type=int, default=2, metavar="G",
                    help="after the timed region, time the same steps with the batch split over G sequence "
                         "groups on their own streams (reported under 'overlap'; 0 or 1: skip)")
    ap.add_argument("--event-every", type=int, default=64, metavar="N",
                    help="bracket the roofline kernel with HIP events in every N-th timed step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--capacity-rows", action="store_true",
                    help="ragged workload: pass verify all B*(k_max+1) allocated target rows instead of "
                         "the sum(k_b+1) rows the verifier scored")
    ap.add_argument("--no-rotate", action="store_true",
                    help="reuse one copy of the logits in every step (by default small workloads rotate "
                         "copies totalling more than 512 MiB)")
    ap.add_argument("--extras", action="store_true",
                    help="also time the drafting sampler (cmsd_draft_sample) and cmsd_confidence_var on the "
                         "drafter rows, after the timed region (reported under 'extras')")
    ap.add_argument("--no-read-ceiling", action="store_true",
                    help="skip the bare-read ceiling (a read of the roofline kernel's rows in its grid "
                         "shape, timed after the timed region)")
    ap.add_argument("--row-shape", default="", metavar="THREADS,DEPTH",
                    help="force the row kernels' workgroup size and loads in flight (cmsd_set_row_shape; "
                         "0 keeps the library's per-launch choice), e.g. 64,3")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run device-to-device copies of MIB MiB (calibrates HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only (asked for --gpus {args.gpus}); the path shards by "
              f"sequence across GPUs with no exchange, so the whole-job figure is N times the one-GPU value",
              file=sys.stderr)
        return 2

    import torch
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(max(1, args.steps)):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": max(1, args.steps)}))
        return 0
    import workloads as W
    from paper_2508_15371_amd import cmsd, pipeline

    cfg = W.CONFIGS[args.workload]
    mode = cmsd.CMSD_MODE_CM if args.mode == "cm" else cmsd.CMSD_MODE_STANDARD
    if args.row_shape:
        cmsd.cmsd_set_row_shape(*(int(x) for x in args.row_shape.split(",")))
    dev = torch.device("cuda:0")
    print(f"[bench] generating {cfg.name} seed {args.seed}", file=sys.stderr, flush=True)
    d = W.generate(cfg, args.seed)

    def up(a):
        if cfg.dtype == "f32":
            return torch.from_numpy(a).to(dev)
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)

    draft, target = up(d["draft"]), up(d["target"])
    drafted = torch.from_numpy(d["drafted"].reshape(-1)).to(dev)
    unif = torch.from_numpy(d["uniforms"].reshape(-1)).to(dev)
    del d
    G = args.streams
    if G < 1 or cfg.B % G:
        print(f"bench.py: --streams must divide B={cfg.B}", file=sys.stderr)
        return 2
    K = cfg.k_max
    prm = pipeline.Params(mode=mode)
    main = torch.cuda.current_stream(dev)

    def make_groups(G):
        # G groups of B/G sequences, each on its own stream: sequences are independent,
        # so the latency-bound tail of one group overlaps the row passes of another
        bg = cfg.B // G
        groups = []
        for g in range(G):
            b0, b1 = g * bg, (g + 1) * bg
            lpg = pipeline.LogitPass(bg, K, cfg.V, dev, prm, dense=not cfg.ragged)
            a = [draft[b0 * K:b1 * K], target[b0 * (K + 1):b1 * (K + 1)], drafted[b0 * K:b1 * K],
                 unif[b0 * (K + 1):b1 * (K + 1)]]
            if cfg.ragged:
                # the verifier scores k_b + 1 positions per sequence, packed by the device
                # offsets: pack the target rows and uniforms once (untimed); every timed
                # step recomputes the same draft lengths from the same drafter rows
                lpg.confidence(a[0], main)
                lpg.draft_len(main)
                a[1] = W.pack_device(a[1], lpg.k, lpg.off, K)
                a[3] = W.pack_device(a[3], lpg.k, lpg.off, K)
                if not args.capacity_rows:
                    # the verifier scored exactly sum(k_b + 1) rows: hand verify that many
                    rt = int(lpg.off[bg].item())
                    a[1], a[3] = a[1][:rt], a[3][:rt]
            groups.append((lpg, a, main if G == 1 else torch.cuda.Stream(dev)))
        # successive steps read different copies of the logits, together more than 512 MiB
        # (twice the 256 MB last-level cache), so no step finds rows a recent one left there
        in_bytes = sum(a[0].nbytes + a[1].nbytes for _, a, _ in groups)
        n_sets = 1 if args.no_rotate else max(1, -(-(512 << 20) // in_bytes))
        sets = [[a] + [[a[0].clone(), a[1].clone(), a[2], a[3]] for _ in range(n_sets - 1)] for _, a, _ in groups]
        torch.cuda.synchronize()
        return groups, sets, n_sets

    groups, sets, n_sets = make_groups(G)
    R_d = cfg.draft_rows
    R_t = (sum(int(lpg.off[cfg.B // G].item()) for lpg, _, _ in groups) if cfg.ragged
           else cfg.dense_target_rows)
    # one cmsd_logit_pass call per step on dense workloads (one stream), else the three calls
    use_fused = args.path == "fused"
    use_pass = args.path == "pass" or (args.path == "auto" and not cfg.ragged)
    if (use_pass or use_fused) and cfg.ragged:
        print(f"bench.py: --path {args.path} needs a dense workload", file=sys.stderr)
        return 2
    if use_fused and G != 1:
        print("bench.py: --path fused runs on one stream", file=sys.stderr)
        return 2
    rk = "k_fused_pass" if use_fused else ("k_row_pass" if use_pass else "k_confidence")

    def step(lpg, a, st, e=None):
        if use_fused:
            # the whole step is the one launch: the events bracket it
            if e is not None:
                e[0].record(st)
            lpg.logit_pass_fused(a[0], a[1], a[2], a[3], st)
            if e is not None:
                e[1].record(st)
            return
        if use_pass:
            lpg.logit_pass(a[0], a[1], a[2], a[3], st, row_events=e)
            return
        if e is not None:
            e[0].record(st)
        lpg.confidence(a[0], st)
        if e is not None:
            e[1].record(st)
        lpg.draft_len(st)
        lpg.verify(a[0], a[1], a[2], a[3], st)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for k in range(args.warmup):
        for gi, (lpg, _, st) in enumerate(groups):
            step(lpg, sets[gi][k % n_sets], st)
    torch.cuda.synchronize()

    # timed region: K steps.  HIP events on the launch stream bracket the roofline
    # kernel (the joint row pass of cmsd_logit_pass, or k_confidence of group 0 on the
    # three-call path) in every `event_every`-th step; each event marker costs time
    # between kernels (and on short steps host time), so no other kernel is bracketed.
    # (the middle step of each block of event_every steps, so never the first timed step,
    # which starts from an idle GPU)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
          if k % args.event_every == min(args.event_every, args.steps) // 2 else None for k in range(args.steps)]
    for e in ev:
        if e is not None:      # the binding hands the library events that exist
            e[0].record(main)
            e[1].record(main)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k, e in enumerate(ev):
        for gi, (lpg, _, st) in enumerate(groups):
            step(lpg, sets[gi][(args.warmup + k) % n_sets], st, e if gi == 0 else None)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / args.steps
    t_roof = float(np.mean([e[0].elapsed_time(e[1]) for e in ev if e is not None])) * 1e-3

    # per-call split, one group after another on one stream (outside the timed region)
    ev2 = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(max(3, args.steps // 4))]
    for i, e in enumerate(ev2):
        cur = [(lpg, sets[gi][i % n_sets]) for gi, (lpg, _, _) in enumerate(groups)]
        e[0].record(main)
        for lpg, a in cur:
            lpg.confidence(a[0], main)
        e[1].record(main)
        for lpg, a in cur:
            lpg.draft_len(main)
        e[2].record(main)
        for lpg, a in cur:
            lpg.verify(a[0], a[1], a[2], a[3], main)
        e[3].record(main)
    torch.cuda.synchronize()
    t_conf1 = float(np.mean([e[0].elapsed_time(e[1]) for e in ev2])) * 1e-3
    t_dl = float(np.mean([e[1].elapsed_time(e[2]) for e in ev2])) * 1e-3
    t_ver = float(np.mean([e[2].elapsed_time(e[3]) for e in ev2])) * 1e-3

    # the same steps with the batch split over `--overlap` sequence groups, each on its
    # own stream, so that one group's final-token kernels overlap another group's row
    # pass (after the timed region, warmed up alike, no events)
    ov = None
    if G == 1 and args.overlap > 1 and cfg.B % args.overlap == 0 and not use_fused:
        print(f"[bench] {args.overlap} stream groups", file=sys.stderr, flush=True)
        g2, s2, n2 = make_groups(args.overlap)
        for k in range(args.warmup):
            for gi, (lpg, _, st) in enumerate(g2):
                step(lpg, s2[gi][k % n2], st)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            for gi, (lpg, _, st) in enumerate(g2):
                step(lpg, s2[gi][(args.warmup + k) % n2], st)
        torch.cuda.synchronize()
        ov = (args.overlap, 1e3 * (time.perf_counter() - t0) / args.steps)
        del g2, s2

    n_acc = np.concatenate([lpg.n_acc.cpu().numpy() for lpg, _, _ in groups])
    k_all = np.concatenate([lpg.k.cpu().numpy() for lpg, _, _ in groups])
    k_used = k_all if cfg.ragged else np.full(cfg.B, cfg.k_max)
    rej = int((n_acc < k_used).sum())
    s = cfg.elem_bytes
    conf_bytes = R_d * cfg.V * s + R_d * 32
    # the roofline kernel's launch (group 0's; the whole batch when G = 1): the joint row
    # pass reads every drafter and target row of the group once and writes a 32-byte
    # record per drafter row, a 32-byte record and a 32-byte slot per target row, after
    # gathering two logits per drafted position; k_confidence reads the group's drafter
    # rows and writes their records
    if use_pass:
        launch_bytes = ((R_d // G) * (cfg.V * s + 32) + (R_t // G) * (cfg.V * s + 64)
                        + (cfg.B // G) * cfg.k_max * 8)
    elif use_fused:
        launch_bytes = None     # the whole step: its algorithmic bytes (below)
    else:
        launch_bytes = (R_d // G) * (cfg.V * s + 32)
    verify_bytes = R_t * cfg.V * s + rej * cfg.V * s + R_t * 32 + cfg.B * cfg.k_max * 8
    step_bytes = conf_bytes + cfg.B * cfg.k_max * 32 + verify_bytes
    if launch_bytes is None:
        launch_bytes = step_bytes

    result = {
        "metric": "logit rows/sec and achieved HBM GB/s (confidence+verify), V=32000-152064",
        "value": (R_d + R_t) / (ms_step * 1e-3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: B={cfg.B} k_max={cfg.k_max} V={cfg.V} {cfg.dtype} "
                               f"{'ragged' if cfg.ragged else 'dense'}, "
                               f"mode={args.mode}", "batch": cfg.B, "k_max": cfg.k_max, "vocab": cfg.V,
                   "drafter_rows": R_d, "target_rows": R_t},
        "gbps_algorithmic": step_bytes / (ms_step * 1e-3) / 1e9,
        "per_call_ms": {"cmsd_confidence": t_conf1 * 1e3, "cmsd_draft_len": t_dl * 1e3, "cmsd_verify": t_ver * 1e3},
        "roofline": {"kernel": rk, "bound": "hbm", "achieved": launch_bytes / t_roof / 1e9,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": launch_bytes / t_roof / 1e9 / PEAK_HBM_GBS,
                     "traffic": _traffic(rk, cfg.name) if G == 1 else None},
        "workload_stats": {"mean_n_acc": float(n_acc.mean()), "rejecting_sequences": rej,
                           "mean_draft_len": float(k_all.mean()), "streams": G,
                           "path": ("cmsd_logit_pass_fused" if use_fused else "cmsd_logit_pass" if use_pass
                                    else "three calls"), "input_copies": n_sets},
    }
    if ov is not None:
        result["overlap"] = {"streams": ov[0], "ms_per_step": ov[1], "value": (R_d + R_t) / (ov[1] * 1e-3),
                             "unit": "rows/s", "gbps_algorithmic": step_bytes / (ov[1] * 1e-3) / 1e9}
    if not args.no_read_ceiling and G == 1 and not use_fused:
        result["read_ceiling"] = read_ceiling(sets, n_sets, cfg, R_t, use_pass, main, args.steps, t_roof)
    if args.extras:
        result["extras"] = extras(cmsd, groups, sets, n_sets, main, cfg, args.steps)
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg.name, args.seed, mode)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
