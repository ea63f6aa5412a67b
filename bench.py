"""Benchmark: Lloyd iterations per second of exact k-means on one MI355X.

Workload: N = 8,388,608 points, D = 128, K = 4,096 centroids, bf16 points with
fp32 accumulation and fp32 centroids, a Zipf(1.1)-weighted Gaussian mixture
(the synthetic stand-in for the paper's token embeddings).  One step = one
Lloyd iteration (assignment + centroid update) through ``kmeans_lloyd``.

Prints one JSON line with the metric, a roofline object for the dominant
kernel (assignment: 2 N K D flops per launch against the dense bf16 MFMA peak)
and the fp64 CPU oracle's rate on the host cores as a reported baseline.
Each fraction is also given against the peak at the clock the GPU ran at
(sampled during the kernel's timing loop) and against ceilings measured in the
same run by microbenchmark kernels (``include/fkm_calib.h``).  The other
workloads (1, 2, 4, 5 and the paper's B = 32 shape) are measured after the
metric workload and reported under ``workloads``.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import statistics
import subprocess
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Lloyd iter/s; assign TFLOP/s as % of MFMA peak at N=8M D=128 K=4096"
PEAK_BF16_TFLOPS = 2516.6          # MI355X dense bf16/fp16 MFMA (no sparsity)
PEAK_F32_TFLOPS = 157.3            # MI355X fp32 MFMA
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E
PEAK_SCLK_MHZ = 2400.0             # the clock the MFMA peaks are quoted at
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "assign_traffic.json")
ASSIGN_SRC = os.path.join(ROOT, "paper_2608_12629_amd", "csrc", "assign_pipe.h")
CALIB_LIB = os.path.join(ROOT, "paper_2608_12629_amd", "libfkm_calib.so")
SCLK_FILES = ["/sys/class/drm/card0/device/pp_dpm_sclk", "/sys/class/drm/card1/device/pp_dpm_sclk"]
EXTRA_WORKLOADS = (1, 2, 4, 5, 6)
FLUSH_BYTES = 512 << 20            # written before each timed sample: evicts L2 and the Infinity Cache


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


# ---------------------------------------------------------------- clock
class SclkSampler:
    """Samples the GPU's current shader clock (the starred level of the
    driver's pp_dpm_sclk table) from a host thread while a timed loop runs."""

    def __init__(self, period_s: float = 0.002):
        self.path = next((p for p in SCLK_FILES if os.path.exists(p)), None)
        self.period = period_s
        self.samples = []
        self._stop = threading.Event()
        self._t = None

    def _read(self):
        try:
            with open(self.path) as f:
                for line in f:
                    if line.rstrip().endswith("*"):
                        return float(line.split(":")[1].strip().split("Mhz")[0].split("MHz")[0])
        except (OSError, ValueError, IndexError):
            return None
        return None

    def _run(self):
        while not self._stop.is_set():
            v = self._read()
            if v is not None:
                self.samples.append(v)
            time.sleep(self.period)

    def __enter__(self):
        if self.path:
            self._t = threading.Thread(target=self._run, daemon=True)
            self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._t:
            self._t.join()

    def median(self):
        # samples taken between kernels (idle levels) are not the running clock
        busy = [s for s in self.samples if s >= 500.0]
        return statistics.median(busy) if busy else None


# ---------------------------------------------------------------- ceilings
def ceilings(torch, X):
    """In-run microbenchmark ceilings: bf16 MFMA with changing operands, a
    streaming read of X, and a random-order gather of X's rows."""
    if not os.path.exists(CALIB_LIB):
        return None
    lib = ctypes.CDLL(CALIB_LIB)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    lib.fkm_calib_mfma.argtypes = [vp, i32, i32, vp]
    lib.fkm_calib_read.argtypes = [vp, sz, vp, i32, vp]
    lib.fkm_calib_gather.argtypes = [vp, i64, i32, vp, i64, vp, i32, vp]
    dev = X.device
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    mfma_blocks, mem_blocks = 512, 4096
    # every kernel writes one word per thread: out holds [blocks * 256] for the largest grid
    out = torch.empty(max(mfma_blocks, mem_blocks) * 256, dtype=torch.float32, device=dev)
    outp = ctypes.c_void_p(out.data_ptr())

    def grid(blocks):
        if blocks * 256 > out.numel():
            raise ValueError(f"{blocks} workgroups write past the {out.numel()}-word output")
        return blocks

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn, reps):
        fn()
        ts = []
        for _ in range(reps):
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    res = {}
    iters = 2000
    with SclkSampler() as sc:
        ms = timed(lambda: lib.fkm_calib_mfma(outp, grid(mfma_blocks), iters, sp), 5)
    flops = mfma_blocks * 4 * iters * 32 * 32768.0
    res["mfma_bf16_TFLOP/s"] = flops / (ms * 1e-3) / 1e12
    res["mfma_sclk_MHz"] = sc.median()
    Xb = X.reshape(-1)
    nbytes = Xb.numel() * Xb.element_size() // 16 * 16
    ms = timed(lambda: lib.fkm_calib_read(ctypes.c_void_p(Xb.data_ptr()), nbytes, outp,
                                          grid(mem_blocks), sp), 5)
    res["read_GB/s"] = nbytes / (ms * 1e-3) / 1e9
    rows = X.shape[0] * X.shape[1]
    row_bytes = X.shape[2] * X.element_size()
    if row_bytes % 16 == 0 and row_bytes <= 1024:
        perm = torch.randperm(rows, device=dev, dtype=torch.int64).to(torch.int32)
        ms = timed(lambda: lib.fkm_calib_gather(ctypes.c_void_p(X.data_ptr()), rows, row_bytes,
                                                ctypes.c_void_p(perm.data_ptr()), rows, outp,
                                                grid(mem_blocks), sp), 5)
        res["gather_GB/s"] = (rows * row_bytes + 4 * rows) / (ms * 1e-3) / 1e9
        del perm
    return res


# ---------------------------------------------------------------- CPU baseline
def cpu_model() -> str:
    """The host CPU's model name with its family/model numbers and logical CPU count."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k = k.strip()
                if k in ("model name", "cpu family", "model") and k not in info:
                    info[k] = v.strip()
    except OSError:
        return "unknown"
    return (f"{info.get('model name', 'unknown')} (family {info.get('cpu family', '?')}, "
            f"model {info.get('model', '?')}, {os.cpu_count()} logical CPUs)")


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
                      f"fp64, OpenMP",
            "cpu_model": cpu_model()}


def oracle_iteration_seconds(index: int) -> float:
    """One full oracle Lloyd iteration (assignment + update) of workload `index`, in this process."""
    from oracle import default
    from paper_2608_12629_amd.synth import make_workload, raw_bits
    w = make_workload(index)
    o = default()
    xr = raw_bits(w.X)
    C64 = w.C0.double().numpy()
    t0 = time.perf_counter()
    o.lloyd(xr, w.dtype, C64, 1)
    return time.perf_counter() - t0


def single_thread_small_f32():
    """The fp64 oracle's full Lloyd iteration of the fp32 workload on one host
    thread (a child process with OMP_NUM_THREADS=1; it does not touch the GPU)."""
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "--oracle-iteration", "1"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        return None
    s = float(r.stdout.strip().splitlines()[-1])
    return {"value": 1.0 / s, "unit": "iter/s", "cores": 1,
            "sample": "one full Lloyd iteration of blobs_n65536_d64_k256_f32 (assignment of all "
                      "points + update), fp64"}


# ---------------------------------------------------------------- KNN
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
    steps = args.steps or 5
    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    samples = []
    with SclkSampler() as sc:
        for _ in range(steps):
            flush.fill_(1)
            torch.cuda.synchronize()
            e0.record(stream)
            km.kmeans_knn(Qd, Rd, k, ni, nd, ws)
            e1.record(stream)
            torch.cuda.synchronize()
            samples.append(e0.elapsed_time(e1))
    del flush
    ms = statistics.median(samples)
    tflops = 2.0 * B * M * N * D / (ms * 1e-3) / 1e12
    sclk = sc.median()
    out = {
        "metric": "KNN search queries/s (k nearest of N rows); distance TFLOP/s as % of MFMA peak",
        "value": B * M / (ms * 1e-3), "unit": "queries/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"knn_m{M}_n{N}_d{D}_k{k}_bf16", "B": B, "M": M, "N": N, "D": D,
                   "k": k, "timing": f"median of {steps} searches, caches flushed before each"},
        "roofline": {"bound": "mfma", "kernel": "knn", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS, "traffic": None},
        "sclk_MHz": sclk,
        "frac_at_sclk": tflops / (PEAK_BF16_TFLOPS * sclk / PEAK_SCLK_MHZ) if sclk else None,
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
                               "kind": "oracle", "cpu_model": cpu_model(),
                               "sample": f"the first {sample} of {M} queries against all {N} rows "
                                         f"({tc:.2f} s); fp64, OpenMP"}
    print(json.dumps(out), flush=True)


# ---------------------------------------------------------------- Lloyd
def measure(torch, km, w, steps, warmup, kernel_reps, reps, graph=True, cold_samples=0):
    """Everything timed for one workload: the host-launched run, per-kernel
    event timings (with the clock sampled meanwhile), optionally cold
    assignments, and `reps` graph replays of `steps` iterations, each after a
    cache flush; the replay median is the workload's rate."""
    dev = torch.device("cuda", 0)
    X = w.X.to(dev)
    C0 = w.C0.to(dev)
    B, N, D, K = w.B, w.N, w.D, w.K
    ws = km.Workspace(B, N, D, K, X.dtype, dev)
    C = C0.clone()
    idx = torch.empty((B, N), dtype=torch.int32, device=dev)
    md = torch.empty((B, N), dtype=torch.float32, device=dev)
    cnt = torch.empty((B, K), dtype=torch.int32, device=dev)
    obj = torch.empty((B, steps), dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()

    # warm-up, then exactly `steps` Lloyd iterations from C0 (host launches)
    km.kmeans_lloyd(X, C, warmup, idx=idx, min_dist=md, counts=cnt, ws=ws)
    C.copy_(C0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    km.kmeans_lloyd(X, C, steps, idx=idx, min_dist=md, counts=cnt, objective=obj, ws=ws)
    torch.cuda.synchronize()
    dt_eager = time.perf_counter() - t0
    C_ref, obj_ref, idx_ref = C.clone(), obj.clone(), idx.clone()

    # per-kernel durations with HIP events on the stream the library launches on
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    with SclkSampler() as sc_assign:
        ev[0].record(stream)
        for _ in range(kernel_reps):
            km.kmeans_assign(X, C0, idx=idx, min_dist=md, ws=ws)
        ev[1].record(stream)
        torch.cuda.synchronize()
    with SclkSampler() as sc_update:
        ev[2].record(stream)
        for _ in range(kernel_reps):
            km.kmeans_update(X, idx, C0, C_out=C, counts=cnt, ws=ws)
        ev[3].record(stream)
        torch.cuda.synchronize()
    assign_ms = ev[0].elapsed_time(ev[1]) / kernel_reps
    update_ms = ev[2].elapsed_time(ev[3]) / kernel_reps

    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    cold = []
    for _ in range(cold_samples):
        flush.fill_(1)
        ev[2].record(stream)
        km.kmeans_assign(X, C0, idx=idx, min_dist=md, ws=ws)
        ev[3].record(stream)
        torch.cuda.synchronize()
        cold.append(ev[2].elapsed_time(ev[3]))

    samples = []
    if graph:
        # the run captured once in a HIP graph, `warmup` untimed replays, then
        # `reps` timed replays of exactly `steps` iterations, each after a
        # cache flush and bracketed by synchronizations; the last is checked
        # bit for bit against the host-launched run
        C.copy_(C0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            km.kmeans_lloyd(X, C, steps, idx=idx, min_dist=md, counts=cnt, objective=obj, ws=ws)
        for _ in range(warmup):
            C.copy_(C0)
            g.replay()
        for _ in range(reps):
            C.copy_(C0)
            flush.fill_(1)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            g.replay()
            torch.cuda.synchronize()
            samples.append(time.perf_counter() - t0)
        if not (torch.equal(C, C_ref) and torch.equal(obj, obj_ref) and torch.equal(idx, idx_ref)):
            raise SystemExit(f"{w.name}: graph replay differs from the host-launched run")
        del g
    else:
        samples = [dt_eager]
    del flush
    dt = statistics.median(samples)

    es = X.element_size()
    flops = 2.0 * B * N * K * D
    peak = PEAK_BF16_TFLOPS if w.dtype != "f32" else PEAK_F32_TFLOPS
    upd_bytes = B * N * D * es + 4 * B * N + 4 * B * K * D + 4 * B * K
    asg_bytes = B * N * D * es + B * K * D * es + 8 * B * N
    res = {
        "iter/s": steps / dt, "ms_per_iter": dt * 1e3 / steps, "steps": steps,
        "iter/s_samples": [steps / s for s in samples],
        "host_launch_ms_per_iter": dt_eager * 1e3 / steps,
        "assign_ms": assign_ms, "update_ms": update_ms,
        "assign_TFLOP/s": flops / (assign_ms * 1e-3) / 1e12,
        "assign_bound": "mfma" if flops / asg_bytes >= peak * 1e12 / (PEAK_HBM_GBS * 1e9) else "hbm",
        "assign_GB/s": asg_bytes / (assign_ms * 1e-3) / 1e9,
        "update_GB/s": upd_bytes / (update_ms * 1e-3) / 1e9,
        "update_algorithmic_bytes": upd_bytes, "assign_algorithmic_bytes": asg_bytes,
        "assign_flops": flops, "mfma_peak": peak,
        "sclk_MHz_assign": sc_assign.median(), "sclk_MHz_update": sc_update.median(),
    }
    if cold:
        res["assign_cold_median_ms"] = statistics.median(cold)
        res["assign_cold_samples"] = len(cold)
    del X, C0, ws, C, idx, md, cnt, obj, C_ref, obj_ref, idx_ref
    return res


def fractions(r, ceil):
    """The assignment's and the update's fractions: of the spec peak, of the
    peak at the sampled clock, and of the in-run ceilings."""
    out = {}
    sa = r.get("sclk_MHz_assign")
    if r["assign_bound"] == "mfma":
        a = r["assign_TFLOP/s"]
        out["assign_frac"] = a / r["mfma_peak"]
        out["assign_frac_at_sclk"] = a / (r["mfma_peak"] * sa / PEAK_SCLK_MHZ) if sa else None
        if ceil and r["mfma_peak"] == PEAK_BF16_TFLOPS:
            out["assign_frac_of_ceiling"] = a / ceil["mfma_bf16_TFLOP/s"]
    else:
        a = r["assign_GB/s"]
        out["assign_frac"] = a / PEAK_HBM_GBS
        if ceil:
            out["assign_frac_of_ceiling"] = a / ceil["read_GB/s"]
    u = r["update_GB/s"]
    out["update_frac"] = u / PEAK_HBM_GBS
    if ceil:
        out["update_frac_of_read_ceiling"] = u / ceil["read_GB/s"]
        if "gather_GB/s" in ceil:
            out["update_frac_of_gather_ceiling"] = u / ceil["gather_GB/s"]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="default: the workload's iterations")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--kernel-reps", type=int, default=10)
    ap.add_argument("--reps", type=int, default=5,
                    help="timed graph replays (each after a cache flush); the median is reported")
    ap.add_argument("--cpu-sample", type=int, default=1 << 20)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-extra", dest="extra", action="store_false",
                    help="skip the other workloads (reported under 'workloads')")
    ap.add_argument("--no-ceilings", dest="ceil", action="store_false",
                    help="skip the in-run microbenchmark ceilings")
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
    ap.add_argument("--oracle-iteration", type=int, default=0, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.oracle_iteration:
        print(oracle_iteration_seconds(args.oracle_iteration), flush=True)
        return
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
    steps = args.steps if args.steps is not None else w.iters

    if args.calib_copy_mib:
        src = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    r = measure(torch, km, w, steps, args.warmup, args.kernel_reps, args.reps, graph=args.graph,
                cold_samples=args.cold_samples)
    log(f"{steps} Lloyd iterations: median {r['ms_per_iter'] * steps:.2f} ms of {len(r['iter/s_samples'])} "
        f"flushed replays ({r['host_launch_ms_per_iter'] * steps:.2f} ms host-launched)")
    log(f"assign {r['assign_ms']:.3f} ms = {r['assign_TFLOP/s']:.1f} TFLOP/s at "
        f"{r['sclk_MHz_assign']} MHz; update {r['update_ms']:.3f} ms = {r['update_GB/s']:.0f} GB/s")
    ceil = None
    if args.ceil:
        X = w.X.to(dev)
        ceil = ceilings(torch, X)
        del X
        log(f"ceilings: {ceil}")
    fr = fractions(r, ceil)

    if r["assign_bound"] == "mfma":
        roofline = {"bound": "mfma", "kernel": "assign", "achieved": r["assign_TFLOP/s"],
                    "peak": r["mfma_peak"], "unit": "TFLOP/s", "frac": fr["assign_frac"],
                    "traffic": stored_traffic(w.name)}
    else:
        roofline = {"bound": "hbm", "kernel": "assign", "achieved": r["assign_GB/s"],
                    "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": fr["assign_frac"],
                    "traffic": stored_traffic(w.name)}
    out = {
        "metric": METRIC,
        "value": r["iter/s"],
        "unit": "iter/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_iter"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "f16": "f16", "f32": "f32"}[w.dtype],
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "D": w.D, "K": w.K, "x_dtype": w.dtype,
                   "centroid_dtype": "f32", "iters_per_step": 1,
                   "launch": "graph replay" if args.graph else "host",
                   "timing": (f"median of {len(r['iter/s_samples'])} timed runs of {steps} "
                              f"iterations, caches flushed before each")},
        "iter/s_samples": r["iter/s_samples"],
        "host_launch_ms_per_step": r["host_launch_ms_per_iter"],
        "roofline": roofline,
        "roofline_more": {
            "sclk_MHz_during_assign": r["sclk_MHz_assign"],
            "assign_frac_at_sclk": fr.get("assign_frac_at_sclk"),
            "assign_frac_of_ceiling": fr.get("assign_frac_of_ceiling"),
            "ceilings": ceil,
        },
        "update": {"ms": r["update_ms"], "algorithmic_bytes": r["update_algorithmic_bytes"],
                   "GB/s": r["update_GB/s"], "hbm_frac": fr["update_frac"],
                   "frac_of_read_ceiling": fr.get("update_frac_of_read_ceiling"),
                   "frac_of_gather_ceiling": fr.get("update_frac_of_gather_ceiling"),
                   "sclk_MHz": r["sclk_MHz_update"]},
        "assign_ms": r["assign_ms"],
        "assign_cold": {"median_ms": r.get("assign_cold_median_ms"),
                        "samples": r.get("assign_cold_samples", 0),
                        "TFLOP/s": (r["assign_flops"] / (r["assign_cold_median_ms"] * 1e-3) / 1e12
                                    if r.get("assign_cold_median_ms") else None)},
    }
    if not args.no_cpu:
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_sample)
        st = single_thread_small_f32()
        if st:
            out["cpu_baseline"]["single_thread"] = st
        log(f"cpu baseline in {time.perf_counter() - t0:.1f} s")
    if args.extra and args.workload == 3:
        # the other workloads at their own sizes and iteration counts (no cold
        # samples, CPU baseline or ceilings of their own)
        del w
        out["workloads"] = {}
        for wl in EXTRA_WORKLOADS:
            t0 = time.perf_counter()
            wx = make_workload(wl)
            rx = measure(torch, km, wx, wx.iters, args.warmup, args.kernel_reps, args.reps,
                         graph=args.graph)
            fx = fractions(rx, ceil)
            out["workloads"][wx.name] = {
                "iter/s": rx["iter/s"], "ms_per_iter": rx["ms_per_iter"], "iters": wx.iters,
                "assign_ms": rx["assign_ms"], "assign_TFLOP/s": rx["assign_TFLOP/s"],
                "assign_bound": rx["assign_bound"], "assign_GB/s": rx["assign_GB/s"],
                "update_ms": rx["update_ms"], "update_GB/s": rx["update_GB/s"],
                "sclk_MHz_assign": rx["sclk_MHz_assign"], **fx}
            log(f"{wx.name}: {rx['iter/s']:.1f} iter/s, assign {rx['assign_ms']:.4f} ms "
                f"({fx['assign_frac']:.3f}), update {rx['update_ms']:.4f} ms "
                f"({fx['update_frac']:.3f}) [{time.perf_counter() - t0:.1f} s]")
            del wx
            torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
