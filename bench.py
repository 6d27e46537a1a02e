"""Benchmark of the SKIP routing core on one MI355X.

One step = one fused route (question pooling -> salience scoring -> top-k
prune -> passage keys -> edge cosines -> edge selection -> sparse
cross-attention) over one synthetic batch already resident in HBM.  The
workload is "highres_bf16": 16 questions, N = 2304 visual tokens of width
4096, k = 192 kept tokens, 10 passages x 256 tokens, 32 heads x 128, average
degree 4 (bf16; selection sums in float64).

Prints ONE JSON line.  ``value`` is queries/s of the whole job.  The timed
steps use the profiled entry point, which records HIP events on the launch
stream between kernel stages; the roofline of the dominant kernel (the
attention) divides its algorithmic bytes by its average event-timed duration.
The CPU baseline times the CPU oracle (single thread) on a few questions of
the same batch.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "queries/sec + fused route TFLOP/s & HBM GB/s vs MI355X peak, N=2304"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="highres_bf16")
    ap.add_argument("--seed", type=int, default=2026)
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="questions of the batch the CPU oracle is timed on (-1, the "
                         "default: the whole batch; 0: skip)")
    ap.add_argument("--no-companion", action="store_true",
                    help="with the default workload, skip the nested mixed_bf16 record")
    ap.add_argument("--avg-degree", type=float, default=None,
                    help="override the workload's average degree (edges per kept row)")
    ap.add_argument("--edge-rule", default="question", choices=["question", "row", "fraction"],
                    help="edge cut: per-question budget (default), per-row top, top fraction")
    ap.add_argument("--edge-metric", default="cosine", choices=["cosine", "dot"],
                    help="edge compatibility: cosine (default) or scaled dot product")
    ap.add_argument("--edge-beta", type=float, default=0.1,
                    help="kept fraction of the pairs for --edge-rule fraction")
    ap.add_argument("--scorer", default="linear", choices=["linear", "mlp"],
                    help="mlp: time the prune stage with the main-text scorer instead of "
                         "the fused route (a record line, not the headline)")
    ap.add_argument("--hidden", type=int, default=512,
                    help="hidden width of the mlp scorer or of the passage gate")
    ap.add_argument("--gate", action="store_true",
                    help="time the fused route with the passage verification gate (and the "
                         "route without it, interleaved) instead of the plain fused route")
    ap.add_argument("--regions", action="store_true",
                    help="time the regions of the kept tokens (k-means of the kept rows, read "
                         "in place through the kept indices) instead of the fused route")
    ap.add_argument("--project", action="store_true",
                    help="time the learned projection of the kept rows (gathered GEMM, rows "
                         "read in place through the kept indices) instead of the fused route")
    ap.add_argument("--proj-out", type=int, default=0,
                    help="output width of the projection (default: d)")
    ap.add_argument("--r-max", type=int, default=8, help="most regions per question")
    ap.add_argument("--kmeans-iter", type=int, default=10, help="Lloyd iterations")
    ap.add_argument("--gate-tau", type=float, default=0.5, help="gate threshold on nu")
    ap.add_argument("--gate-rho", type=float, default=0.5,
                    help="kept fraction of a question's passages after the gate")
    ap.add_argument("--cold", action="store_true",
                    help="overwrite a 1 GiB buffer before every timed step so that no input "
                         "is left in the on-die cache; value then comes from the event-timed "
                         "median step")
    ap.add_argument("--pass-keys", action="store_true",
                    help="hand precomputed passage keys to the library (skips pooling)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip measuring the box's streaming and GEMM ceilings")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run an elementwise copy (negation) of MIB MiB of "
                         "float32 three times, so a hardware-counter pass can scale "
                         "FETCH_SIZE / WRITE_SIZE by a kernel of known traffic")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_sparse_kernel.highres_bf16.traffic.json")
ATTN_SOURCE = os.path.join(ROOT, "paper_2607_25422_amd", "csrc", "attn.hip")


def measure_ceilings(torch) -> dict:
    """Attainable rates on this GPU, beside the published peaks: an elementwise
    copy (negation, 1 GiB in and out), a column sum reading 1 GiB of bf16, and
    a 16384^3 bf16 GEMM (hipBLASLt through torch.matmul)."""
    def timed(fn, it):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(it):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / it
    n = 1 << 30
    a = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    copy = 2 * n / timed(lambda: torch.neg(a, out=b), 10) / 1e9
    del a, b
    c = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda").view(-1, 4096)
    read = n / timed(lambda: c.sum(0, dtype=torch.float32), 10) / 1e9
    del c
    m = 16384
    x = torch.randn(m, m, dtype=torch.bfloat16, device="cuda")
    y = torch.randn(m, m, dtype=torch.bfloat16, device="cuda")
    gemm = 2 * m ** 3 / timed(lambda: x @ y, 5) / 1e12
    del x, y
    torch.cuda.empty_cache()
    return {"copy_gbs": round(copy, 1), "read_gbs": round(read, 1),
            "gemm_bf16_tflops": round(gemm, 1),
            "what": "negation copy of 1 GiB float32; column sum of 1 GiB bf16; "
                    "16384^3 bf16 GEMM (torch.matmul)"}


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed counter summary, or
    None when it was taken on another workload or an older attention source."""
    import hashlib
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    sha = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
    if rec.get("workload") != workload or rec.get("attn_source_sha256") != sha:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def bench_mlp_scorer(args):
    """Prune stage (pooling, main-text scorer, top-k, gather) on a workload's
    visual tokens: queries/s of the stage and the scorer's first-layer
    TFLOP/s over the whole stage time (event-timed on the launch stream)."""
    import torch

    from paper_2607_25422_amd import binding as B
    from paper_2607_25422_amd import workloads as wls

    torch.cuda.set_device(0)
    print(f"[bench] generating {args.workload} seed {args.seed} (scorer h={args.hidden})",
          file=sys.stderr, flush=True)
    batch = wls.make_batch(args.workload, args.seed, threads=16)
    wl = batch.wl
    w = wls.make_scorer_weights(wl, args.hidden, args.seed)
    db = B.to_device(batch)
    p = db.p
    mlp = B.QvsMlp(w.W1.cuda(), w.b1.cuda(), w.w2.cuda(), w.b2)
    ws = torch.empty(B.workspace_bytes_mlp(p, args.hidden), dtype=torch.uint8, device="cuda")
    for _ in range(args.warmup):
        B.prune_topk_mlp(db, mlp, want_scores=False, workspace=ws)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        B.prune_topk_mlp(db, mlp, want_scores=False, workspace=ws)
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    avg_ms = sum(step_ms) / len(step_ms)
    flops = 2.0 * p.B * p.N * (2 * p.d) * args.hidden + 2.0 * p.B * args.hidden * p.d
    tf = flops / (avg_ms * 1e-3) / 1e12
    res = {
        "metric": "queries/sec (prune stage with the main-text scorer) + scorer TFLOP/s vs "
                  "MI355X bf16 MFMA peak",
        "value": round(p.B * args.steps / wall, 1),
        "unit": "queries/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "B": p.B, "N": p.N, "d": p.d, "k": int(batch.k[0]),
                   "scorer": "mlp", "hidden": args.hidden, "seed": args.seed},
        "step_gpu_ms": {"p10": round(step_ms[len(step_ms) // 10], 5),
                        "p50": round(step_ms[len(step_ms) // 2], 5),
                        "p90": round(step_ms[min(len(step_ms) - 1, 9 * len(step_ms) // 10)], 5)},
        "roofline": {"kernel": "mlp_score_kernel (over the whole stage)", "bound": "mfma",
                     "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "algorithmic_gflop": round(flops / 1e9, 2), "avg_ms": round(avg_ms, 5)},
    }
    print(json.dumps(res), flush=True)


def bench_gated_route(args):
    """The fused route with the verification step (score, top-k, gate, graph
    on the verified passages, attention) against the plain fused route,
    alternating step by step on the same batch, plus the gate call alone on
    the gathered rows with the passage keys handed over as float32 (its
    algorithmic bytes: question tokens, kept rows, the gate weights and the
    keys, each read once)."""
    import torch

    from paper_2607_25422_amd import binding as B
    from paper_2607_25422_amd import workloads as wls

    torch.cuda.set_device(0)
    print(f"[bench] generating {args.workload} seed {args.seed} (gate h={args.hidden})",
          file=sys.stderr, flush=True)
    batch = wls.make_batch(args.workload, args.seed, threads=16)
    wl = batch.wl
    w = wls.make_gate_weights(wl, args.hidden, args.seed)
    db = B.to_device(batch)
    p = db.p
    g = B.SkvGate(w.W.cuda(), w.b1.cuda(), w.w2.cuda(), w.b2, args.gate_tau, args.gate_rho)
    ws = torch.empty(B.workspace_bytes_gate(p, args.hidden), dtype=torch.uint8, device="cuda")
    dev = "cuda"
    gout = (torch.empty(p.total_kept, dtype=torch.int32, device=dev),
            torch.empty(p.total_passages, dtype=torch.uint8, device=dev),
            torch.empty(p.total_passages, dtype=torch.float32, device=dev),
            torch.empty((p.total_kept, p.H, p.d_h), dtype=batch.torch_dtype, device=dev),
            torch.empty((p.total_kept, p.H), dtype=torch.float32, device=dev))
    pout = (gout[0], gout[3], gout[4])
    _, _, Vk = B.prune_topk(db, want_scores=False)
    pk = torch.stack([batch.Kh[a:b].float().reshape(b - a, -1).mean(0) for a, b in
                      zip(batch.passage_offsets[:-1], batch.passage_offsets[1:])]).cuda()
    for _ in range(args.warmup):
        B.route_fused_gated(db, g, out=gout, workspace=ws)
        B.route_fused(db, out=pout)
        B.skv_gate(db, g, Vk, passage_keys=pk, workspace=ws)
    torch.cuda.synchronize()
    kept = int(gout[1].sum())
    n = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n)]
    t_gated = 0.0
    for i in range(n):
        ev[i][0].record()
        B.route_fused_gated(db, g, out=gout, workspace=ws)
        ev[i][1].record()
        B.route_fused(db, out=pout)
        ev[i][2].record()
        B.skv_gate(db, g, Vk, passage_keys=pk, workspace=ws)
        ev[i][3].record()
    torch.cuda.synchronize()
    gated = sorted(e[0].elapsed_time(e[1]) for e in ev)
    plain = sorted(e[1].elapsed_time(e[2]) for e in ev)
    gate_only = sorted(e[2].elapsed_time(e[3]) for e in ev)
    mean = lambda xs: sum(xs) / len(xs)   # noqa: E731
    # wall-clock throughput of the gated route alone
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        B.route_fused_gated(db, g, out=gout, workspace=ws)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    h, d = args.hidden, p.d
    gate_bytes = (p.total_qtok * d * 2 + p.total_kept * d * 2 + h * 5 * d * 2
                  + p.total_passages * d * 4 + 4 * h * 2 + p.total_passages * 5)
    gate_flops = 2.0 * p.total_passages * h * 3 * d + 2.0 * p.B * h * 2 * d
    gms = mean(gate_only)
    gbs = gate_bytes / (gms * 1e-3) / 1e9
    res = {
        "metric": "queries/sec (fused route with the passage verification gate) + gate-call "
                  "HBM GB/s vs MI355X peak",
        "value": round(p.B * n / wall, 1),
        "unit": "queries/s",
        "n_gpus": 1, "steps": n, "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / n, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "B": p.B, "N": p.N, "d": p.d,
                   "passages": int(batch.P[0]), "gate_hidden": h, "tau": args.gate_tau,
                   "rho": args.gate_rho, "seed": args.seed},
        "gated_route_gpu_ms": {"p50": round(gated[n // 2], 5), "mean": round(mean(gated), 5)},
        "plain_route_gpu_ms": {"p50": round(plain[n // 2], 5), "mean": round(mean(plain), 5)},
        "passages_kept": kept, "passages": p.total_passages,
        "roofline": {"kernel": "skip_skv_gate call (3 kernels, keys given)", "bound": "hbm",
                     "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes": gate_bytes, "avg_ms": round(gms, 5),
                     "gflop": round(gate_flops / 1e9, 3)},
    }
    print(json.dumps(res), flush=True)


FP64_PEAK_TFLOPS = 78.6


def bench_project(args):
    """Learned projection Y = W x_r of every kept row (rows read in place
    through the kept indices of a prune call made beforehand): the timed
    steps are the one-call form (W repacked inside the call); the roofline is
    the GEMM alone, from the same projection with W packed once beforehand,
    event-timed on the launch stream: 2 * M * d * d_out FLOP per call against
    the bf16 matrix peak."""
    import torch

    from paper_2607_25422_amd import binding as B
    from paper_2607_25422_amd import workloads as wls

    torch.cuda.set_device(0)
    print(f"[bench] generating {args.workload} seed {args.seed} (projection)", file=sys.stderr,
          flush=True)
    batch = wls.make_batch(args.workload, args.seed, threads=16)
    wl = batch.wl
    db = B.to_device(batch)
    p = db.p
    d_out = args.proj_out or p.d
    W = wls.make_projection(d_out, p.d, args.seed).cuda()
    idx, _, _ = B.prune_topk(db, want_scores=False, want_rows=False)
    ws = torch.empty(B.workspace_bytes_project(p, d_out), dtype=torch.uint8, device="cuda")
    Y = torch.empty((p.total_kept, d_out), dtype=torch.bfloat16, device="cuda")
    run = lambda: B.skip_gather_project(p, db.V, db.kept_offsets, idx, W, Y,  # noqa: E731
                                        workspace=ws)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    n = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(n):
        run()
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(n))
    avg = sum(ms) / n
    flops = 2.0 * p.total_kept * p.d * d_out
    tf = flops / (avg * 1e-3) / 1e12
    # the same projection with W packed once beforehand: the GEMM kernel alone
    packed = B.pack_projection(db, W)
    run_p = lambda: B.skip_gather_project_packed(p, db.V, db.kept_offsets, idx,  # noqa: E731
                                                 packed, d_out, Y)
    for _ in range(args.warmup):
        run_p()
    torch.cuda.synchronize()
    evp = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    evp[0].record()
    for i in range(n):
        run_p()
        evp[i + 1].record()
    torch.cuda.synchronize()
    avg_p = sum(evp[i].elapsed_time(evp[i + 1]) for i in range(n)) / n
    tf_p = flops / (avg_p * 1e-3) / 1e12
    res = {
        "metric": "queries/sec (learned projection of the kept rows) + bf16 TFLOP/s vs MI355X "
                  "bf16 MFMA peak",
        "value": round(p.B * n / wall, 1),
        "unit": "queries/s",
        "n_gpus": 1, "steps": n, "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / n, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "B": p.B, "rows": p.total_kept, "d": p.d,
                   "d_out": d_out, "seed": args.seed},
        "step_gpu_ms": {"p10": round(ms[n // 10], 5), "p50": round(ms[n // 2], 5),
                        "p90": round(ms[min(n - 1, 9 * n // 10)], 5)},
        "roofline": {"kernel": "proj_gemm_kernel (weights packed once beforehand)",
                     "bound": "mfma", "achieved": round(tf_p, 1), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tf_p / BF16_PEAK_TFLOPS, 4),
                     "traffic": None, "algorithmic_gflop": round(flops / 1e9, 2),
                     "avg_ms": round(avg_p, 5)},
        "one_call": {"what": "skip_gather_project: repack of W + GEMM, the timed steps",
                     "avg_ms": round(avg, 5), "tflops": round(tf, 1)},
        "packed_call": {"what": "skip_gather_project_packed after skip_pack_projection",
                        "avg_ms": round(avg_p, 5), "tflops": round(tf_p, 1),
                        "queries_per_s": round(p.B / (avg_p * 1e-3), 1)},
    }
    print(json.dumps(res), flush=True)


def bench_regions(args):
    """Regions of the kept tokens: k-means of each question's kept rows (read
    in place through the kept indices of a prune call made beforehand),
    event-timed on the launch stream.  The floor is the float64 arithmetic of
    the assignment: 2 * k * R * d FLOP per question and iteration."""
    import torch

    from paper_2607_25422_amd import binding as B
    from paper_2607_25422_amd import workloads as wls

    torch.cuda.set_device(0)
    print(f"[bench] generating {args.workload} seed {args.seed} (regions)", file=sys.stderr,
          flush=True)
    batch = wls.make_batch(args.workload, args.seed, threads=16)
    wl = batch.wl
    db = B.to_device(batch)
    p = db.p
    idx, _, _ = B.prune_topk(db, want_scores=False, want_rows=False)
    ws = torch.empty(B.workspace_bytes_regions(p, args.r_max), dtype=torch.uint8, device="cuda")
    for _ in range(args.warmup):
        B.region_kmeans(db, db.V, kept_idx=idx, r_max=args.r_max, n_iter=args.kmeans_iter,
                        workspace=ws)
    torch.cuda.synchronize()
    n = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(n):
        B.region_kmeans(db, db.V, kept_idx=idx, r_max=args.r_max, n_iter=args.kmeans_iter,
                        workspace=ws)
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(n))
    avg = sum(ms) / n
    R = [max(1, min(int(k) // 4, args.r_max)) if k > 0 else 0 for k in batch.k]
    flops = sum(2.0 * int(k) * r * p.d for k, r in zip(batch.k, R)) * args.kmeans_iter
    tf = flops / (avg * 1e-3) / 1e12
    res = {
        "metric": "queries/sec (regions of the kept tokens, k-means) + float64 TFLOP/s vs "
                  "MI355X fp64 peak",
        "value": round(p.B * n / wall, 1),
        "unit": "queries/s",
        "n_gpus": 1, "steps": n, "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / n, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": wl.name, "B": p.B, "d": p.d,
                   "k": int(batch.k[0]) if len(set(batch.k.tolist())) == 1 else "mixed",
                   "r_max": args.r_max, "iterations": args.kmeans_iter, "seed": args.seed},
        "step_gpu_ms": {"p10": round(ms[n // 10], 5), "p50": round(ms[n // 2], 5),
                        "p90": round(ms[min(n - 1, 9 * n // 10)], 5)},
        "roofline": {"kernel": "region_step_kernel (over the whole call)", "bound": "alu",
                     "achieved": round(tf, 2), "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / FP64_PEAK_TFLOPS, 4), "traffic": None,
                     "algorithmic_gflop": round(flops / 1e9, 3), "avg_ms": round(avg, 5)},
    }
    print(json.dumps(res), flush=True)


def measure_route(args, workload):
    """The fused route on one workload: `steps` timed steps (after `warmup`),
    then a profiled pass with stage events.  Returns (record, batch, device
    batch, passage keys or None, average degree)."""
    import numpy as np
    import torch

    from paper_2607_25422_amd import accounting as acc
    from paper_2607_25422_amd import binding as B
    from paper_2607_25422_amd import workloads as wls

    print(f"[bench] generating {workload} seed {args.seed}", file=sys.stderr, flush=True)
    batch = wls.make_batch(workload, args.seed, threads=16)
    wl = batch.wl
    db = B.to_device(batch, avg_degree=args.avg_degree, edge_rule=args.edge_rule,
                     edge_metric=args.edge_metric, edge_beta=args.edge_beta)
    p = db.p
    avg_degree = wl.avg_degree if args.avg_degree is None else args.avg_degree
    elem = 4 if wl.dtype == "f32" else 2
    pkeys = None
    if args.pass_keys:
        # passage keys as a retriever would hand them over (mean of the keys)
        pk = torch.stack([batch.Kh[a:b].float().reshape(b - a, -1).mean(0) for a, b in
                          zip(batch.passage_offsets[:-1], batch.passage_offsets[1:])])
        pkeys = pk.cuda()

    # The graph, once, outside the timed region: realised edges for the FLOP
    # and byte accounting.
    idx, _, Vk = B.prune_topk(db, want_scores=False)
    _, _, rp, col = B.bipartite_xattn(db, Vk.view(-1, p.H, p.d_h), passage_keys=pkeys)
    torch.cuda.synchronize()
    rp_h, col_h = rp.cpu().numpy(), col.cpu().numpy()
    edge_L = acc.edge_lengths_from_csr(rp_h, col_h, batch.kept_offsets, batch.query_passages,
                                       batch.passage_offsets)
    touched = acc.touched_passages(rp_h, col_h, batch.kept_offsets, batch.query_passages)
    L = np.diff(batch.passage_offsets)
    touched_tokens = int(L[touched].sum()) if touched.size else 0
    attn_flops = acc.attention_flops(edge_L, p.H, p.d_h)
    attn_bytes = acc.attention_bytes(p.total_kept, p.d, p.H, touched_tokens, elem, elem)
    score_bytes = acc.score_bytes(p.B, p.N, p.d, elem)
    route_bytes = acc.route_bytes(p.B, p.N, p.d, p.total_qtok, p.total_kept, p.H,
                                  p.total_tokens, touched_tokens, elem, pooled_keys=pkeys is None)
    del idx, Vk, rp, col

    out = (torch.empty(p.total_kept, dtype=torch.int32, device="cuda"),
           torch.empty((p.total_kept, p.H, p.d_h), dtype=batch.torch_dtype, device="cuda"),
           torch.empty((p.total_kept, p.H), dtype=torch.float32, device="cuda"))
    if args.calibrate_copy > 0:
        src = torch.ones(args.calibrate_copy << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        B.route_fused(db, passage_keys=pkeys, out=out)
    torch.cuda.synchronize()
    print(f"[bench] warmup done; timing {args.steps} steps", file=sys.stderr, flush=True)

    # Timed region: exactly `steps` fused routes and nothing else on the
    # stream.  With --cold a 1 GiB fill overwrites the last-level cache before
    # every step; it is not part of a step, so each step is then bracketed by
    # its own pair of events and the median step gives the rate.
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda") if args.cold else None
    cold_ev = ([(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(args.steps)] if args.cold else None)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if flush is not None:
            flush.fill_(float(i))
            cold_ev[i][0].record()
        B.route_fused(db, passage_keys=pkeys, out=out)
        if flush is not None:
            cold_ev[i][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    if args.cold:
        cold_ms = sorted(a.elapsed_time(b) for a, b in cold_ev)
        ms_per_step = cold_ms[len(cold_ms) // 2]
        qps = p.B / (ms_per_step * 1e-3)
    else:
        ms_per_step = 1e3 * wall / args.steps
        qps = p.B * args.steps / wall

    # Profiled pass, after the timed region and not part of it: the same
    # routes with an event between every two kernel stages (the stage split,
    # the attention time of the roofline, per-step percentiles).  Each event
    # on the stream costs a few microseconds, so these steps run longer than
    # the timed ones.
    n_prof = min(args.steps, 50)
    events = [B.StageEvents() for _ in range(n_prof)]
    for i in range(n_prof):
        if flush is not None:
            flush.fill_(float(i))
        B.route_fused(db, passage_keys=pkeys, out=out, stage_events=events[i])
    torch.cuda.synchronize()
    stages = {k: 0.0 for k in B.FUSED_STAGES}
    step_ms = []
    for ev in events:
        sm = ev.stage_ms()
        step_ms.append(sum(sm.values()))
        for k, v in sm.items():
            stages[k] += v / n_prof
    gpu_ms = sum(stages.values())
    step_sorted = sorted(step_ms)

    def pct(q):
        return step_sorted[min(len(step_sorted) - 1, int(q * len(step_sorted)))]

    attn_ms = stages["attention"]
    attn_gbs = attn_bytes / (attn_ms * 1e-3) / 1e9
    # The prune stage on its own: question pooling, then scoring and top-k in
    # one launch (skip_prune_topk without scores or gathered rows), events
    # around each call.  In the fused route the same scoring launch also
    # pools the passage keys, so its "score" stage holds both streams.
    pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n_prof)]
    for _ in range(3):
        B.prune_topk(db, want_scores=False, want_rows=False)
    for e0, e1 in pev:
        e0.record()
        B.prune_topk(db, want_scores=False, want_rows=False)
        e1.record()
    torch.cuda.synchronize()
    prune_ms = sorted(a.elapsed_time(b) for a, b in pev)[n_prof // 2]
    score_gbs = score_bytes / (prune_ms * 1e-3) / 1e9

    res = {
        "metric": METRIC,
        "value": round(qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "B": p.B, "N": p.N, "d": p.d, "T": wl.T,
                   "k": int(batch.k[0]) if len(set(batch.k.tolist())) == 1 else "mixed",
                   "passages": int(batch.P[0]) if len(set(batch.P.tolist())) == 1 else "mixed",
                   "L_p": wl.L_p, "H": p.H, "d_h": p.d_h, "avg_degree": avg_degree,
                   "seed": args.seed, "passage_keys": "given" if pkeys is not None else "pooled",
                   "cache": "cold" if args.cold else "warm", "edge_rule": args.edge_rule,
                   "edge_metric": args.edge_metric,
                   **({"edge_beta": args.edge_beta} if args.edge_rule == "fraction" else {})},
        "step_gpu_ms": {"p10": round(pct(0.1), 5), "p50": round(pct(0.5), 5),
                        "p90": round(pct(0.9), 5), "steps": n_prof,
                        "what": "profiled pass: stage events on the stream, after the timed steps"},
        "roofline": {
            "kernel": "attn_sparse_kernel" if wl.dtype == "bf16" else "attn_f32_kernel",
            "bound": "hbm",
            "achieved": round(attn_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl.name),
            "algorithmic_bytes": attn_bytes,
            "avg_ms": round(attn_ms, 5),
        },
        "attention": {
            "tflops": round(attn_flops / (attn_ms * 1e-3) / 1e12, 2),
            "mfma_peak_frac": round(attn_flops / (attn_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "algorithmic_gflop": round(attn_flops / 1e9, 3),
            "edges": int(rp_h[-1]),
        },
        "prune": {
            "ms": round(prune_ms, 5),
            "what": "question pooling + scoring with top-k (skip_prune_topk), median of "
                    "event-timed calls",
            "score_gbs": round(score_gbs, 1),
            "score_hbm_frac": round(score_gbs / HBM_PEAK_GBS, 4),
        },
        "route": {
            "gpu_ms": round(gpu_ms, 5),
            "algorithmic_bytes": route_bytes,
            "gbs": round(route_bytes / (gpu_ms * 1e-3) / 1e9, 1),
            "tflops": round(attn_flops / (gpu_ms * 1e-3) / 1e12, 2),
        },
        "stages_ms": {k: round(v, 5) for k, v in stages.items()},
    }

    return res, batch, db, pkeys, avg_degree


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the routing core runs on a single MI355X; see the sharding notes)",
              file=sys.stderr)
        sys.exit(2)
    if args.scorer == "mlp":
        bench_mlp_scorer(args)
        return
    if args.gate:
        bench_gated_route(args)
        return
    if args.regions:
        bench_regions(args)
        return
    if args.project:
        bench_project(args)
        return

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    res, batch, db, pkeys, avg_degree = measure_route(args, args.workload)
    wl, p = batch.wl, db.p
    if args.workload == "highres_bf16" and not args.no_companion:
        # the other N = 2304 configuration, in the same run: the difficulty-
        # mixed batch, nested as a record of its own
        comp, cbatch, cdb, _, _ = measure_route(args, "mixed_bf16")
        res["mixed_bf16"] = {k: comp[k] for k in ("value", "unit", "ms_per_step", "config",
                                                  "roofline", "attention", "prune",
                                                  "stages_ms", "step_gpu_ms")}
        del cbatch, cdb
        torch.cuda.empty_cache()

    if not args.no_ceilings:
        ceil = measure_ceilings(torch)
        res["ceilings"] = ceil
        res["roofline"]["frac_of_read_ceiling"] = round(
            res["roofline"]["achieved"] / ceil["read_gbs"], 4)
        res["prune"]["score_frac_of_read_ceiling"] = round(
            res["prune"]["score_gbs"] / ceil["read_gbs"], 4)

    if args.cpu_sample != 0:
        from threadpoolctl import threadpool_limits

        import oracle as orc
        n_q = p.B if args.cpu_sample < 0 else min(args.cpu_sample, p.B)
        qs = list(range(n_q))
        # as many BLAS threads as the process may run on
        cores = len(os.sched_getaffinity(0))
        print(f"[bench] timing the CPU oracle on {len(qs)} questions, {cores} threads",
              file=sys.stderr, flush=True)
        with threadpool_limits(cores):
            c0 = time.perf_counter()
            orc.route(batch.V, batch.Qtok, batch.q_offsets, batch.kept_offsets, batch.Kh,
                      batch.Vh, batch.passage_offsets, batch.query_passages, wl.scale,
                      avg_degree, passage_key_table=None if pkeys is None else pkeys.cpu(),
                      queries=qs, edge_rule=args.edge_rule, edge_metric=args.edge_metric,
                      edge_beta=args.edge_beta)
            c1 = time.perf_counter()
        res["cpu_baseline"] = {
            "value": round(len(qs) / (c1 - c0), 4),
            "unit": "queries/s",
            "cores": cores,
            "kind": "oracle",
            "sample": (f"{len(qs)} of {p.B} questions of {wl.name} seed {args.seed}: full route "
                       f"(pooling, scoring, top-k, graph, attention of every kept row), float64 "
                       f"numpy, {cores} BLAS threads, {c1 - c0:.1f} s"),
            "cpu": cpu_model(),
        }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
