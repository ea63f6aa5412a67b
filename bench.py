"""Benchmark: Lloyd iterations per second of exact k-means on one MI355X.

Workload: N = 8,388,608 points, D = 128, K = 4,096 centroids, bf16 points with
fp32 accumulation and fp32 centroids, a Zipf(1.1)-weighted Gaussian mixture
(the synthetic stand-in for the paper's token embeddings).  One step = one
Lloyd iteration (assignment + centroid update) through ``kmeans_lloyd``.

Prints one JSON line with the metric, a roofline object for the dominant
kernel (assignment: 2 N K D flops per launch against the dense bf16 MFMA peak)
and the fp64 CPU oracle's rate on the host cores as a reported baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import statistics
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Lloyd iter/s; assign TFLOP/s as % of MFMA peak at N=8M D=128 K=4096"
PEAK_BF16_TFLOPS = 2516.6          # MI355X dense bf16/fp16 MFMA (no sparsity)
PEAK_F32_TFLOPS = 157.3            # MI355X fp32 MFMA
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "assign_traffic.json")
ASSIGN_SRC = os.path.join(ROOT, "paper_2608_12629_amd", "csrc", "assign_pipe.h")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    with open(ASSIGN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def stored_traffic(workload: str):
    """Measured HBM bytes per assignment launch, if taken on this workload and
    the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("kernel_sha256_16") != kernel_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(w, sample_rows: int):
    """The fp64 oracle on the host: one Lloyd iteration, assignment timed on a row sample."""
    import numpy as np
    from oracle import default
    from paper_2608_12629_amd.synth import raw_bits

    o = default()
    xr = raw_bits(w.X)
    C64 = w.C0.double().numpy()
    n = min(sample_rows, w.N)  # rows of each instance
    rows = np.ascontiguousarray(xr[:, :n])
    t0 = time.perf_counter()
    idx_s, _, _ = o.assign(rows, w.dtype, C64)
    t_assign = time.perf_counter() - t0
    # the update is O(N D): time it in full, on an assignment of every point
    idx_full = np.resize(idx_s, (w.B, w.N)).astype(np.int32)
    t0 = time.perf_counter()
    o.update(xr, w.dtype, idx_full, C64)
    t_update = time.perf_counter() - t0
    t_iter = t_assign * (w.N / n) + t_update
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    what = f"all {w.N} points" if n == w.N else f"the first {n} of {w.N} points"
    inst = f" of each of {w.B} instances" if w.B > 1 else ""
    scaled = "" if n == w.N else f", scaled by N/{n}"
    return {"value": 1.0 / t_iter, "unit": "iter/s", "cores": cores, "kind": "oracle",
            "sample": f"assignment of {what}{inst} against all {w.K} centroids "
                      f"({t_assign:.2f} s{scaled}) + the full update ({t_update:.2f} s); "
                      f"fp64, OpenMP"}


def knn_bench(args):
    """KNN search (queries/s) on synthetic blobs; one JSON line like the Lloyd bench."""
    import torch
    from paper_2608_12629_amd import kmeans as km

    B, M, N, D, k = 1, args.knn_queries, args.knn_rows, 128, args.knn_k
    g = torch.Generator().manual_seed(7)
    centres = torch.rand((N // 64, D), generator=g) * 2 - 1
    R = (centres[torch.randint(0, N // 64, (N,), generator=g)] + 0.1 * torch.randn((N, D), generator=g))
    Q = (centres[torch.randint(0, N // 64, (M,), generator=g)] + 0.1 * torch.randn((M, D), generator=g))
    R, Q = R.to(torch.bfloat16), Q.to(torch.bfloat16)
    dev = torch.device("cuda", 0)
    Qd, Rd = Q.to(dev), R.to(dev)
    ni = torch.empty((B, M, k), dtype=torch.int32, device=dev)
    nd = torch.empty((B, M, k), dtype=torch.float32, device=dev)
    ws = torch.empty(km.knn_workspace_bytes(B, M, N, D, k, torch.bfloat16), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        km.kmeans_knn(Qd, Rd, k, ni, nd, ws)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps or 5):
        km.kmeans_knn(Qd, Rd, k, ni, nd, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    steps = args.steps or 5
    ms = e0.elapsed_time(e1) / steps
    tflops = 2.0 * B * M * N * D / (ms * 1e-3) / 1e12
    out = {
        "metric": "KNN search queries/s (k nearest of N rows); distance TFLOP/s as % of MFMA peak",
        "value": B * M * steps / dt, "unit": "queries/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": dt * 1e3 / steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"knn_m{M}_n{N}_d{D}_k{k}_bf16", "B": B, "M": M, "N": N, "D": D, "k": k},
        "roofline": {"bound": "mfma", "kernel": "knn", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS, "traffic": None},
    }
    if not args.no_cpu:
        import numpy as np
        from oracle import default
        from paper_2608_12629_amd.synth import raw_bits
        o = default()
        sample = min(M, args.knn_cpu_queries)
        qs = np.ascontiguousarray(raw_bits(Q[None, :sample]))
        t0 = time.perf_counter()
        o.knn(qs, raw_bits(R[None]), "bf16", k)
        tc = time.perf_counter() - t0
        cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        out["cpu_baseline"] = {"value": sample / tc, "unit": "queries/s", "cores": cores,
                               "kind": "oracle",
                               "sample": f"the first {sample} of {M} queries against all {N} rows "
                                         f"({tc:.2f} s); fp64, OpenMP"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="default: the workload's iterations")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--kernel-reps", type=int, default=10)
    ap.add_argument("--cpu-sample", type=int, default=1 << 20)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--workload", type=int, default=3,
                    help="1..6; 3 (N=8M, D=128, K=4096) is the metric workload, 6 the "
                         "paper's B=32 assignment shape (context)")
    ap.add_argument("--cold-samples", type=int, default=5,
                    help="assignments timed one by one after evicting the caches (median reported)")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="time the host-launched Lloyd run instead of its graph replay")
    ap.add_argument("--knn", action="store_true", help="measure the KNN search instead")
    ap.add_argument("--knn-queries", type=int, default=262144)
    ap.add_argument("--knn-rows", type=int, default=1 << 20)
    ap.add_argument("--knn-k", type=int, default=10)
    ap.add_argument("--knn-cpu-queries", type=int, default=1536)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(rerun with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.knn:
        knn_bench(args)
        return

    import torch
    from paper_2608_12629_amd import kmeans as km
    from paper_2608_12629_amd.synth import make_workload

    t0 = time.perf_counter()
    w = make_workload(args.workload)
    log(f"workload {w.name} generated in {time.perf_counter() - t0:.1f} s")
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    X = w.X.to(dev)
    C0 = w.C0.to(dev)
    B, N, D, K = w.B, w.N, w.D, w.K
    if args.steps is None:
        args.steps = w.iters
    ws = km.Workspace(B, N, D, K, X.dtype, dev)
    C = C0.clone()
    idx = torch.empty((B, N), dtype=torch.int32, device=dev)
    md = torch.empty((B, N), dtype=torch.float32, device=dev)
    cnt = torch.empty((B, K), dtype=torch.int32, device=dev)

    if args.calib_copy_mib:
        src = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # warm-up, then exactly `steps` Lloyd iterations from C0 (host launches)
    obj = torch.empty((B, args.steps), dtype=torch.float64, device=dev)
    km.kmeans_lloyd(X, C, args.warmup, idx=idx, min_dist=md, counts=cnt, ws=ws)
    C.copy_(C0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    km.kmeans_lloyd(X, C, args.steps, idx=idx, min_dist=md, counts=cnt, objective=obj, ws=ws)
    torch.cuda.synchronize()
    dt = dt_eager = time.perf_counter() - t0
    log(f"{args.steps} Lloyd iterations in {dt * 1e3:.2f} ms (host launches)")
    C_ref, obj_ref, idx_ref = C.clone(), obj.clone(), idx.clone()

    # per-kernel durations with HIP events on the stream the library launches on
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    ev[0].record(stream)
    for _ in range(args.kernel_reps):
        km.kmeans_assign(X, C0, idx=idx, min_dist=md, ws=ws)
    ev[1].record(stream)
    for _ in range(args.kernel_reps):
        km.kmeans_update(X, idx, C0, C_out=C, counts=cnt, ws=ws)
    ev[2].record(stream)
    torch.cuda.synchronize()
    assign_ms = ev[0].elapsed_time(ev[1]) / args.kernel_reps
    update_ms = ev[1].elapsed_time(ev[2]) / args.kernel_reps
    flops = 2.0 * B * N * K * D
    assign_tflops = flops / (assign_ms * 1e-3) / 1e12
    # cold-cache samples: a 512 MB write evicts L2 and the Infinity Cache
    # before each timed assignment; the median is reported beside the mean
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold = []
    for _ in range(args.cold_samples):
        flush.fill_(1)
        ev[2].record(stream)
        km.kmeans_assign(X, C0, idx=idx, min_dist=md, ws=ws)
        ev[3].record(stream)
        torch.cuda.synchronize()
        cold.append(ev[2].elapsed_time(ev[3]))
    del flush
    cold_ms = statistics.median(cold) if cold else None
    if args.graph:
        # the same run captured once in a HIP graph: `warmup` untimed replays,
        # then one timed replay of exactly `steps` iterations, checked bit for
        # bit against the host-launched run (timed after the kernels, so that
        # the kernel timings run under the same conditions either way)
        C.copy_(C0)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            km.kmeans_lloyd(X, C, args.steps, idx=idx, min_dist=md, counts=cnt, objective=obj,
                            ws=ws)
        for _ in range(args.warmup):
            C.copy_(C0)
            graph.replay()
        C.copy_(C0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        graph.replay()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        log(f"{args.steps} Lloyd iterations in {dt * 1e3:.2f} ms (graph replay)")
        if not (torch.equal(C, C_ref) and torch.equal(obj, obj_ref) and torch.equal(idx, idx_ref)):
            raise SystemExit("graph replay differs from the host-launched run")
        del graph, C_ref, obj_ref, idx_ref
    upd_bytes = B * N * D * X.element_size() + 4 * B * N + 4 * B * K * D + 4 * B * K
    peak = PEAK_BF16_TFLOPS if w.dtype != "f32" else PEAK_F32_TFLOPS
    upd_gbs = upd_bytes / (update_ms * 1e-3) / 1e9
    # the assignment's bound: MFMA above the ridge (peak flops / HBM bandwidth),
    # HBM below it (small K: its bytes are X once, the centroids, idx and min_dist)
    asg_bytes = B * N * D * X.element_size() + B * K * D * X.element_size() + 8 * B * N
    if flops / asg_bytes >= peak * 1e12 / (PEAK_HBM_GBS * 1e9):
        roofline = {"bound": "mfma", "kernel": "assign", "achieved": assign_tflops, "peak": peak,
                    "unit": "TFLOP/s", "frac": assign_tflops / peak,
                    "traffic": stored_traffic(w.name)}
    else:
        asg_gbs = asg_bytes / (assign_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": "assign", "achieved": asg_gbs, "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": asg_gbs / PEAK_HBM_GBS,
                    "traffic": stored_traffic(w.name)}
    log(f"assign {assign_ms:.3f} ms = {assign_tflops:.1f} TFLOP/s; "
        f"update {update_ms:.3f} ms = {upd_gbs:.0f} GB/s algorithmic")

    out = {
        "metric": METRIC,
        "value": args.steps / dt,
        "unit": "iter/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "f16": "f16", "f32": "f32"}[w.dtype],
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "N": N, "D": D, "K": K, "x_dtype": w.dtype,
                   "centroid_dtype": "f32", "iters_per_step": 1,
                   "launch": "graph replay" if args.graph else "host"},
        "host_launch_ms_per_step": dt_eager * 1e3 / args.steps,
        "roofline": roofline,
        "update": {"ms": update_ms, "algorithmic_bytes": upd_bytes, "GB/s": upd_gbs,
                   "hbm_frac": upd_gbs / PEAK_HBM_GBS},
        "assign_ms": assign_ms,
        "assign_cold": {"median_ms": cold_ms, "samples": len(cold),
                        "TFLOP/s": flops / (cold_ms * 1e-3) / 1e12 if cold_ms else None},
    }
    if not args.no_cpu:
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample)
        log(f"cpu baseline in {time.perf_counter() - t0:.1f} s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
