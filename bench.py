"""Benchmark of the out-of-core CSR x CSR product (GCN aggregation, after
AIRES arXiv 2507.02006) on one MI355X.

A step is one pass of the whole path over the workload with inputs
resident in HBM: RoBW planning (aires_tile_plan), row analysis, binning,
symbolic phase, scan, the nnz read-back, C allocation, numeric phase
(aires_spgemm), until C is ready on the stream.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload 3] [--cpu-seconds S]
  python bench.py --workload 2 --combine 256    (the combination step, Eq. 3)
  python bench.py --workload 3 --dense-h 256    (aggregation with dense features)

value  = whole-job GFLOP/s (2 flops per intermediate product) per step.
roofline = the dominant kernel (the numeric launch with the largest time):
  achieved = its algorithmic bytes per launch / its average launch time,
  from HIP events the library records around that launch on the compute
  stream during the timed steps.
cpu_baseline = the CPU oracle (serial) on a bounded random row sample;
cpu_baseline_all_cores = the same oracle calls over all host cores.
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

HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
METRIC = "SpGEMM GFLOP/s and achieved HBM GB/s (% of peak) on 1 MI355X; end-to-end latency"

WORKLOAD_NAMES = {
    1: "tiny GCN aggregation: symmetric R-MAT(.57,.19,.19,.05) n=4096 deg 16 + self-loops, sym-normalised; "
       "X 4096x256 10% U(-1,1)",
    2: "mid GCN aggregation: symmetric R-MAT n=262144 deg 32 + self-loops, sym-normalised; X 262144x512 5% U(-1,1)",
    3: "two-hop square A*A: symmetric R-MAT n=1048576 deg 16 + self-loops, sym-normalised fp32 CSR",
    4: "large GCN aggregation: symmetric R-MAT n=8388608 deg 24 + self-loops; X 8388608x128 10% U(-1,1)",
}

KIND_NAMES = ["empty", "dense_wave", "dense_block", "hash_128", "hash_1024", "hash_8192", "windows", "split",
              "hash_4096"]


def row_kinds(P: np.ndarray, N: int) -> np.ndarray:
    """The library's default row bins (aires.cpp bin_plan) for the byte model."""
    k = np.zeros(len(P), dtype=np.int8)
    if N <= 2048:
        k[(P > 0) & (P <= 8192)] = 1
        k[(P > 8192) & (P <= 65536)] = 2
        k[P > 65536] = 7
    else:
        k[(P > 0) & (P <= 64)] = 3
        k[(P > 64) & (P <= 512)] = 4
        k[(P > 512) & (P <= 2048)] = 8
        k[(P > 2048) & (P <= 4096)] = 5
        k[P > 4096] = 6 if N > 16384 else 2
    return k


def row_products(A, B) -> np.ndarray:
    lenB = np.diff(B.rp.astype(np.int64))
    rows = np.repeat(np.arange(A.nrows), np.diff(A.rp.astype(np.int64)))
    return np.bincount(rows, weights=lenB[A.col], minlength=A.nrows).astype(np.int64)


def cpu_baseline(A, B, P, seconds: float, seed: int = 7, threads: int = 1):
    """Time the CPU oracle on random contiguous row ranges whose products add
    up to about `seconds` of work per thread (rate probed on a first small
    range); one oracle call per range, the ranges spread over `threads` host
    threads (the C oracle runs outside the GIL)."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    rng = np.random.default_rng(seed)
    cumr = np.concatenate([[0], np.cumsum(P)])
    total = int(cumr[-1])

    def ranges(nprod, parts):
        out = []
        for st in rng.integers(0, A.nrows, parts):
            en = int(np.searchsorted(cumr, cumr[st] + nprod / parts)) + 1
            out.append((int(st), min(A.nrows, max(en, int(st) + 1))))
        return out

    def span(rg):
        return oracle.spgemm(A, B, rg[0], rg[1]).products

    t0 = time.perf_counter()
    p0 = span(ranges(min(2_000_000, total), 1)[0])
    rate = p0 / max(time.perf_counter() - t0, 1e-9)
    rgs = ranges(min(rate * seconds * threads, total), threads * 4)
    t0 = time.perf_counter()
    if threads == 1:
        prods = sum(span(r) for r in rgs)
    else:
        with ThreadPoolExecutor(threads) as ex:
            prods = sum(ex.map(span, rgs))
    dt = time.perf_counter() - t0
    return {
        "value": round(2 * prods / dt / 1e9, 4),
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "%d random contiguous row ranges (seed %d), %d intermediate products = %.2f%% of the "
                  "workload, %.1f s on %d thread(s)" % (len(rgs), seed, prods, 100.0 * prods / max(total, 1),
                                                        dt, threads),
    }


def host_cpu():
    """Host CPU model and the cores this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def traffic_sources_sha256() -> str:
    """SHA-256 over kernels.hip followed by aires.cpp."""
    import hashlib
    h = hashlib.sha256()
    for name in ("kernels.hip", "aires.cpp"):
        with open(os.path.join(ROOT, "paper_2507_02006_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel_name: str, dom_bytes_launch: int):
    """HBM bytes per launch of the dominant kernel, from the committed
    rocprofv3 FETCH_SIZE/WRITE_SIZE summary (profiles/traffic.json), only
    if it was taken on the kernels and the planner (whose defaults shape
    the launches) as they are now; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
        sha = traffic_sources_sha256()
    except OSError:
        return None
    ent = rec.get(kernel_name)
    if not ent or ent.get("sources_sha256") != sha:
        return None
    return int(ent["traffic_bytes"])


def spmm_kernels(algo, nnz, m, k):
    """Kernel names aires_spmm launches for `algo` (its AUTO rule: dense
    tiles from one entry in eight)."""
    dense = algo == "dense_tiles" or (algo == "auto" and 8 * nnz >= m * k and k <= 1 << 20)
    return "k_spmm_dense" if dense else "k_spmm_rows + k_spmm_heavy"


def spmm_roofline(algo, m, k, F, nnz, flops, compulsory, gather, launch_ms):
    """Entry gather: HBM-bound on the compulsory bytes (C, W once, Y).
    Dense tiles: bound by the fp32 matrix cores on the m*K*F multiply-adds
    they execute (the product's own 2*nnz*F flops beside it)."""
    kern = spmm_kernels(algo, nnz, m, k)
    sec = launch_ms * 1e-3
    if kern == "k_spmm_dense":
        dense_flops = 2.0 * m * k * F
        return {"bound": "mfma", "kernel": kern, "achieved": round(dense_flops / sec / 1e12, 3),
                "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(dense_flops / sec / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                "algorithmic_flops": dense_flops, "avg_launch_ms": round(launch_ms, 4),
                "product_tflops": round(flops / sec / 1e12, 3),
                "compulsory_gbs": round(compulsory / sec / 1e9, 2)}
    return {"bound": "hbm", "kernel": kern, "achieved": round(compulsory / sec / 1e9, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(compulsory / sec / 1e9 / HBM_PEAK_GBS, 4), "traffic": None,
            "algorithmic_bytes": compulsory, "avg_launch_ms": round(launch_ms, 4),
            "gather_model_gbs": round(gather / sec / 1e9, 2), "fp32_tflops": round(flops / sec / 1e12, 3)}


def combine(args, A, B, dA, dB, gen_s):
    """The combination step relu(C W) on the aggregated features C = A B."""
    import torch
    import paper_2507_02006_amd as aires
    F = args.combine
    with aires.tile_plan(dA, dB, 0) as plan:
        C = aires.spgemm(plan)
        torch.cuda.synchronize()
    Cd = (C.nrows, C.ncols, C.rp, C.col, C.val)
    g = torch.Generator(device="cuda").manual_seed(17)
    W = (torch.rand((C.ncols, F), generator=g, device="cuda") - 0.5) / float(np.sqrt(C.ncols))
    Y = torch.empty((C.nrows, F), dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        aires.spmm(Cd, W, relu=True, out=Y, algo=args.spmm_algo)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t_start = time.perf_counter()
    for e0, e1 in ev:
        e0.record()
        aires.spmm(Cd, W, relu=True, out=Y, algo=args.spmm_algo)
        e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = 1e3 * elapsed / args.steps
    launch_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    nnz, m = int(C.nnz), int(C.nrows)
    flops = 2.0 * nnz * F
    compulsory = 8 * (m + 1) + 8 * nnz + 4 * C.ncols * F + 4 * m * F  # C, W once, Y
    gather = 8 * (m + 1) + 8 * nnz + 4 * nnz * F + 4 * m * F          # a row of W per entry of C
    res = {
        "metric": "SpMM GFLOP/s of the GCN combination step relu(C W) (Eq. 3) on 1 MI355X",
        "value": round(flops / (ms_per_step * 1e-3) / 1e9, 3),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded R-MAT graph and uniform sparse features; uniform random weights)",
        "config": {"workload": "combination of cfg%d %s: C (%d x %d, %d nnz) times W (%d x %d), ReLU"
                               % (args.workload, WORKLOAD_NAMES[args.workload], m, C.ncols, nnz, C.ncols, F),
                   "m": m, "k": int(C.ncols), "f_out": F, "nnz_c": nnz, "parallelism": "single GPU"},
        "roofline": spmm_roofline(args.spmm_algo, m, int(C.ncols), F, nnz, flops, compulsory, gather, launch_ms),
        "generation_s": round(gen_s, 2),
    }
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_combine_baseline(C, W, args.cpu_seconds)
    print(json.dumps(res), flush=True)


def cpu_combine_baseline(C, W, seconds):
    """The oracle's double-precision product on leading row blocks of C,
    one core, until about `seconds` of work."""
    import oracle
    from workloads import CSR
    rp = C.rp.cpu().numpy()
    Wn = W.cpu().numpy()
    F = Wn.shape[1]
    col, val = C.col.cpu().numpy(), C.val.cpu().numpy()
    done = 0
    t0 = time.perf_counter()
    r0 = 0
    while time.perf_counter() - t0 < seconds and r0 < C.nrows:
        r1 = min(C.nrows, r0 + 4096)
        blk = CSR(r1 - r0, C.ncols, rp[r0:r1 + 1] - rp[r0], col[rp[r0]:rp[r1]], val[rp[r0]:rp[r1]])
        oracle.spmm(blk, Wn, relu=True)
        done += int(rp[r1] - rp[r0])
        r0 = r1
    dt = time.perf_counter() - t0
    return {"value": round(2.0 * done * F / dt / 1e9, 4), "unit": "GFLOP/s", "cores": 1, "kind": "oracle",
            "sample": "leading rows of C in blocks of 4096: %d of %d entries = %.2f%% of the workload, %.1f s"
                      % (done, int(C.nnz), 100.0 * done / max(1, int(C.nnz)), dt)}


def dense_aggregate(args, A, dA, gen_s):
    """Y = A_norm * H for a dense H (aires_spmm without activation)."""
    import torch
    import paper_2507_02006_amd as aires
    F = args.dense_h
    g = torch.Generator(device="cuda").manual_seed(19)
    H = torch.rand((A.ncols, F), generator=g, device="cuda") * 2 - 1
    Y = torch.empty((A.nrows, F), dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        aires.spmm(dA, H, out=Y, algo=args.spmm_algo)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t_start = time.perf_counter()
    for e0, e1 in ev:
        e0.record()
        aires.spmm(dA, H, out=Y, algo=args.spmm_algo)
        e1.record()
    torch.cuda.synchronize()
    ms_per_step = 1e3 * (time.perf_counter() - t_start) / args.steps
    launch_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    nnz, m, sA = int(A.nnz), int(A.nrows), A.rp.dtype.itemsize
    flops = 2.0 * nnz * F
    compulsory = sA * (m + 1) + 8 * nnz + 4 * A.ncols * F + 4 * m * F  # A, H once, Y
    gather = sA * (m + 1) + 8 * nnz + 4 * nnz * F + 4 * m * F          # a row of H per entry of A
    res = {
        "metric": "SpMM GFLOP/s of the aggregation A_norm H with dense features (Eq. 1) on 1 MI355X",
        "value": round(flops / (ms_per_step * 1e-3) / 1e9, 3),
        "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded R-MAT graph; uniform random dense features)",
        "config": {"workload": "cfg%d graph (%d nodes, %d nnz) times dense H (%d x %d)"
                               % (args.workload, m, nnz, A.ncols, F),
                   "m": m, "k": int(A.ncols), "f": F, "nnz_a": nnz, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": spmm_kernels(args.spmm_algo, nnz, m, int(A.ncols)),
                     "achieved": round(gather / (launch_ms * 1e-3) / 1e9, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gather / (launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None, "algorithmic_bytes": gather, "avg_launch_ms": round(launch_ms, 4),
                     "compulsory_gbs": round(compulsory / (launch_ms * 1e-3) / 1e9, 2)},
        "generation_s": round(gen_s, 2),
    }
    print(json.dumps(res), flush=True)


def streamed(args):
    """Out-of-core aggregation (Alg. 2): A and X in pinned host memory, row-block
    tiles streamed to HBM double-buffered and C tiles returned to pinned host
    memory, under each device budget of --budget-gb and each feature width of
    --features (analogues of the paper's budget and feature-size studies).
    One JSON line per (width, budget); each line's steps are whole calls,
    planning included, with the host C allocation."""
    import torch
    import workloads
    import paper_2507_02006_amd as aires
    cfg = workloads.CONFIGS[args.workload]
    if cfg["F"] is None:
        sys.exit("bench.py --stream: workload %d is not a feature aggregation" % args.workload)
    n = args.nodes or cfg["n"]
    feats = [int(x) for x in args.features.split(",")] if args.features else [cfg["F"]]
    budgets = [float(x) for x in args.budget_gb.split(",")] if args.budget_gb else [32.0]
    segs = args.segmentation.split(",")
    hold = []

    def pinned(rp_dtype):
        def out(nnz):
            rp = torch.empty(n + 1, dtype=rp_dtype, pin_memory=True)
            col = torch.empty(max(nnz, 1), dtype=torch.int32, pin_memory=True)[:nnz]
            val = torch.empty(max(nnz, 1), dtype=torch.float32, pin_memory=True)[:nnz]
            hold.append((rp, col, val))
            return rp.numpy(), col.numpy(), val.numpy()
        return out

    t0 = time.perf_counter()
    A = workloads.rmat_sym(n, cfg["deg"], seed=args.workload, rp64=cfg["rp64"],
                           out=pinned(torch.int64 if cfg["rp64"] else torch.int32), verbose=True)
    tA = (A.nrows, A.ncols) + hold[-1]
    gen_a = time.perf_counter() - t0
    meta = None
    if args.storage:
        # A on storage: its arrays written once into a file, then each call
        # reads every tile from it (direct I/O) before sending it
        t1 = time.perf_counter()
        meta = workloads.write_csr_file(os.path.join(args.storage, "aires_a_cfg%d.csr" % args.workload), A)
        os.sync()
        print("[stream] A written to %s in %.1f s" % (meta["path"], time.perf_counter() - t1), file=sys.stderr,
              flush=True)
    for F in feats:
        t0 = time.perf_counter()
        B = workloads.features(n, F, cfg["rho"], seed=1000 + args.workload, out=pinned(torch.int32), verbose=True)
        tB = (B.nrows, B.ncols) + hold[-1]
        gen_s = gen_a + time.perf_counter() - t0
        meta_b = None
        if meta is not None:
            # B on storage too: read whole into HBM at the start of each call
            meta_b = workloads.write_csr_file(os.path.join(args.storage, "aires_b_cfg%d_f%d.csr" % (args.workload, F)),
                                              B)
            os.sync()
        for budget, seg in [(b, sg) for b in budgets for sg in segs]:
            runs = []
            for it in range(args.warmup + args.steps):
                t1 = time.perf_counter()
                a_in = tA[:4] + (None,) if args.sym_norm else tA
                b_read = None
                if meta is not None:
                    Bd, b_read = aires.read_csr_file(meta_b, mem="device")
                    b_dev = (B.nrows, B.ncols, Bd.rp, Bd.col, Bd.val)
                    plan_cm = aires.tile_plan_file(meta, b_dev, int(budget * (1 << 30)), c_on_host=not args.c_on_device,
                                                   timing=True, max_tile_bytes=args.max_tile_mb << 20,
                                                   a_values="sym_norm" if args.sym_norm else "given")
                else:
                    plan_cm = aires.tile_plan(a_in, tB, int(budget * (1 << 30)), c_on_host=not args.c_on_device,
                                              timing=True, max_tile_bytes=args.max_tile_mb << 20,
                                              a_values="sym_norm" if args.sym_norm else "given",
                                              c_bound=3 if args.c_bound == "rows" else 0, segmentation=seg)
                with plan_cm as plan:
                    t2 = time.perf_counter()
                    info = aires.plan_info(plan)
                    C = aires.spgemm(plan)
                    torch.cuda.synchronize()
                    t3 = time.perf_counter()
                    st = aires.plan_stats(plan)
                    st["_plan_ms"], st["_call_ms"] = 1e3 * (t2 - t1), 1e3 * (t3 - t2)
                    t4 = time.perf_counter()
                    if C.on_host:
                        C.free()
                    del C
                    st["_free_ms"] = 1e3 * (time.perf_counter() - t4)
                st["_b_read"] = b_read
                if b_read is not None:
                    del Bd, b_dev
                wall = time.perf_counter() - t1
                if it >= args.warmup:
                    runs.append((wall, st))
                print("[stream] F=%d budget=%.1f GB %s run %d: %.1f ms, %d tiles" %
                      (F, budget, seg, it, 1e3 * wall, info.ntiles), file=sys.stderr, flush=True)
            walls = sorted(r[0] for r in runs)
            wall = walls[len(walls) // 2]
            st = [r[1] for r in runs if r[0] == wall][0]
            compute = sum(st[k] for k in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms"))
            flops = 2.0 * st["products"]
            res = {
                "metric": "SpGEMM GFLOP/s end to end, A and X streamed from pinned host memory (Alg. 2) "
                          "on 1 MI355X",
                "value": round(flops / wall / 1e9, 3), "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps,
                "warmup": args.warmup, "ms_per_step": round(1e3 * wall, 2), "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": "f32",
                "data": "synthetic (seeded R-MAT graph and uniform sparse features, in pinned host memory)",
                "config": {"workload": "cfg%d-shaped streamed aggregation: n=%d, X %d x %d at %g" %
                                       (args.workload, n, n, F, cfg["rho"]),
                           "budget_gb": budget, "f": F, "nnz_a": A.nnz, "nnz_b": B.nnz, "segmentation": seg,
                           "a_values": "derived on the device (Eq. 2)" if args.sym_norm else "copied",
                           "c_placement": "device" if args.c_on_device else "pinned host",
                           "c_bound": "rows" if meta is not None else args.c_bound,
                           "c_bound_entries": info.c_bound_entries,
                           "a_source": "file (direct I/O)" if meta is not None else "pinned host memory",
                           "b_source": "file (direct I/O), read whole into HBM through pinned staging at the "
                                       "start of the call" if meta is not None else "pinned host memory",
                           "products": st["products"], "nnz_c": st["nnz_c"], "tiles": info.ntiles,
                           "peak_device_gb": round(info.peak_bytes / 1e9, 2), "parallelism": "single GPU"},
                "plan_ms": round(st["_plan_ms"], 2), "call_ms": round(st["_call_ms"], 2),
                "free_c_ms": round(st["_free_ms"], 2), "library_total_ms": round(st["total_ms"], 2),
                "pipeline_ms": round(st["pipeline_ms"], 2), "h2d_ms": round(st["h2d_ms"], 2),
                "d2h_ms": round(st["d2h_ms"], 2), "compute_ms": round(compute, 2),
                "parts_in_sequence_ms": round(st["h2d_ms"] + compute + st["d2h_ms"], 2),
                "h2d_gb": round(st["h2d_bytes"] / 1e9, 3), "d2h_gb": round(st["d2h_bytes"] / 1e9, 3),
                "h2d_gbs": round(st["h2d_bytes"] / max(st["h2d_ms"], 1e-9) / 1e6, 2),
                "d2h_gbs": round(st["d2h_bytes"] / max(st["d2h_ms"], 1e-9) / 1e6, 2),
                "resent_gb": round(st["resent_bytes"] / 1e9, 4), "merge_ms": round(st["merge_ms"], 2),
                "storage_gb": round(st["storage_bytes"] / 1e9, 3), "storage_read_ms": round(st["storage_ms"], 2),
                "storage_gbs": round(st["storage_bytes"] / max(st["storage_ms"], 1e-9) / 1e6, 2),
                "host_syncs": st["host_syncs"],
                "generation_s": round(gen_s, 2),
            }
            if st["_b_read"] is not None:
                br = st["_b_read"]
                res.update({"b_read_ms": round(br["total_ms"], 2), "b_read_gb": round(br["bytes_read"] / 1e9, 3),
                            "b_read_gbs": round(br["bytes_read"] / max(br["total_ms"], 1e-9) / 1e6, 2),
                            "b_storage_read_ms": round(br["read_ms"], 2)})
            print(json.dumps(res), flush=True)
        if meta_b is not None:
            os.unlink(meta_b["path"])
        del B, tB
        hold.pop()
    if meta is not None:
        os.unlink(meta["path"])


def in_core_run(A, B, dA, dB, steps, warmup):
    """Time `steps` whole in-core steps (plan + spgemm until C is ready, C
    dropped) after `warmup`; per-phase and per-kind times from the library's
    HIP events; the dominant numeric launch against the HBM roofline."""
    import torch
    import paper_2507_02006_amd as aires
    P = row_products(A, B)
    total_products = int(P.sum())

    def step():
        with aires.tile_plan(dA, dB, 0, timing=True) as plan:
            C = aires.spgemm(plan)
            torch.cuda.synchronize()
            st = aires.plan_stats(plan)
        return C, st

    for _ in range(warmup):
        C, _ = step()
        del C
    torch.cuda.synchronize()
    stats = []
    t_start = time.perf_counter()
    for _ in range(steps):
        C, st = step()
        stats.append(st)
        last_rp = C.rp  # only the row pointers outlive the step, as for a caller that consumes C
        del C
    torch.cuda.synchronize()
    ms_per_step = 1e3 * (time.perf_counter() - t_start) / steps
    assert all(s["products"] == total_products for s in stats)
    nnz_c = stats[-1]["nnz_c"]
    # dominant kernel: numeric launch of the kind with the largest time
    num_ms = {k: np.mean([s["kind_ms"]["numeric"][k] for s in stats]) for k in KIND_NAMES}
    dom = max(num_ms, key=num_ms.get)
    kinds = row_kinds(P, B.ncols)
    sel = kinds == KIND_NAMES.index(dom)
    crow = np.diff(last_rp.cpu().numpy())
    alen = np.diff(A.rp.astype(np.int64))
    sA = A.rp.dtype.itemsize
    dom_bytes = int((sA + 8 * alen[sel] + 8 + 8 * crow[sel]).sum()) + B.nbytes()
    dom_gbs = dom_bytes / (num_ms[dom] * 1e-3) / 1e9
    # gather model (no reuse): B.row_ptr per A entry and 8 bytes of B per product
    sB = B.rp.dtype.itemsize
    dom_gather = int((sA + 8 * alen[sel] + 2 * sB * alen[sel] + 8 * P[sel] + 8 + 8 * crow[sel]).sum())
    phase = {k: round(float(np.mean([s[k] for s in stats])), 4)
             for k in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms", "total_ms")}
    compulsory = A.nbytes() + B.nbytes() + 8 * (A.nrows + 1) + 8 * nnz_c
    return {
        "ms_per_step": ms_per_step, "P": P, "products": total_products, "nnz_c": nnz_c,
        "tiles": stats[-1]["ntiles"], "dominant": dom,
        "roofline": {"bound": "hbm", "kernel": "numeric/%s" % dom, "achieved": round(dom_gbs, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dom_gbs / HBM_PEAK_GBS, 4),
                     "traffic": None, "algorithmic_bytes": dom_bytes, "avg_launch_ms": round(num_ms[dom], 4),
                     "gather_model_gbs": round(dom_gather / (num_ms[dom] * 1e-3) / 1e9, 2)},
        "phases_ms": phase,
        "numeric_gflops": round(2 * total_products / (phase["numeric_ms"] * 1e-3) / 1e9, 2),
        "end_to_end_compulsory_gbs": round(compulsory / (ms_per_step * 1e-3) / 1e9, 2),
        "numeric_kind_ms": {k: round(float(v), 4) for k, v in num_ms.items() if v > 0},
    }


def overlap_fraction(ts, a="h2d", b="compute"):
    """Share of the busy time of phase `a` (summed over tiles) during which
    phase `b` of some tile was running, from the per-tile event instants."""
    ia = [(t[a + "_begin_ms"], t[a + "_end_ms"]) for t in ts if t[a + "_begin_ms"] >= 0]
    ib = [(t[b + "_begin_ms"], t[b + "_end_ms"]) for t in ts if t[b + "_begin_ms"] >= 0]
    busy = sum(e - s for s, e in ia)
    if busy <= 0:
        return None
    both = sum(max(0.0, min(e1, e2) - max(s1, s2)) for s1, e1 in ia for s2, e2 in ib)
    return round(both / busy, 4)


def extras(args):
    """The other configurations in the same record: cfg2 in core (the
    bench's step, same timing rules), and cfg5 as the out-of-core call of
    Algorithm 2 (A and X generated into pinned host memory, a 32 GB device
    budget, C returned to pinned host memory; whole calls, planning and the
    host C allocation included)."""
    import torch
    import workloads
    import paper_2507_02006_amd as aires
    from paper_2507_02006_amd import _binding as B_
    out = {}
    t0 = time.perf_counter()
    A, B = workloads.workload(2)
    gen = time.perf_counter() - t0
    dA, dB = aires.to_device(A), aires.to_device(B)
    r = in_core_run(A, B, dA, dB, 10, 3)
    out["cfg2_in_core"] = {
        "workload": "cfg2 " + WORKLOAD_NAMES[2], "products": r["products"], "nnz_c": r["nnz_c"],
        "ms_per_step": round(r["ms_per_step"], 4),
        "gflops": round(2 * r["products"] / (r["ms_per_step"] * 1e-3) / 1e9, 3),
        "numeric_gflops": r["numeric_gflops"], "phases_ms": r["phases_ms"],
        "dominant_kernel": r["roofline"]["kernel"], "dominant_ms": r["roofline"]["avg_launch_ms"],
        "dominant_frac_hbm": r["roofline"]["frac"], "dominant_gbs": r["roofline"]["achieved"],
        "steps": 10, "warmup": 3, "generation_s": round(gen, 2)}
    print("[bench] cfg2 in core: %.3f ms" % r["ms_per_step"], file=sys.stderr, flush=True)
    del dA, dB, A, B
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    cfg = workloads.CONFIGS[5]
    n = cfg["n"]
    hold = []

    def pinned(rp_dtype):
        def alloc(nnz):
            rp = torch.empty(n + 1, dtype=rp_dtype, pin_memory=True)
            col = torch.empty(max(nnz, 1), dtype=torch.int32, pin_memory=True)[:nnz]
            val = torch.empty(max(nnz, 1), dtype=torch.float32, pin_memory=True)[:nnz]
            hold.append((rp, col, val))
            return rp.numpy(), col.numpy(), val.numpy()
        return alloc

    t0 = time.perf_counter()
    A = workloads.rmat_sym(n, cfg["deg"], seed=5, rp64=True, out=pinned(torch.int64))
    B = workloads.features(n, cfg["F"], cfg["rho"], seed=1005, out=pinned(torch.int32))
    gen = time.perf_counter() - t0
    print("[bench] cfg5 generated in %.1f s" % gen, file=sys.stderr, flush=True)
    tA, tB = (A.nrows, A.ncols) + hold[0], (B.nrows, B.ncols) + hold[1]
    budget = 32 << 30

    def calls(c_bound):
        runs = []
        for it in range(1 + 3):
            t1 = time.perf_counter()
            with aires.tile_plan(tA, tB, budget, c_on_host=True, timing=True, c_bound=c_bound) as plan:
                t2 = time.perf_counter()
                info = aires.plan_info(plan)
                C = aires.spgemm(plan)
                torch.cuda.synchronize()
                t3 = time.perf_counter()
                st = aires.plan_stats(plan)
                ts = aires.plan_tile_stats(plan)
                peak = plan.allocator.peak
                C.free()
                del C
            wall = time.perf_counter() - t1
            print("[bench] cfg5 streamed call %d (c_bound %d): %.1f ms" % (it, c_bound, 1e3 * wall),
                  file=sys.stderr, flush=True)
            if it >= 1:
                runs.append((wall, 1e3 * (t2 - t1), 1e3 * (t3 - t2), st, ts, peak, info))
        runs.sort(key=lambda x: x[0])
        wall, plan_ms, call_ms, st, ts, peak, info = runs[len(runs) // 2]
        compute = sum(st[k] for k in ("analyze_ms", "bin_ms", "symbolic_ms", "scan_ms", "numeric_ms"))
        return {
            "budget_gb": 32, "tiles": info.ntiles, "products": st["products"], "nnz_c": st["nnz_c"],
            "c_bound_entries": info.c_bound_entries,
            "end_to_end_ms": round(1e3 * wall, 2), "plan_ms": round(plan_ms, 2), "call_ms": round(call_ms, 2),
            "pipeline_ms": round(st["pipeline_ms"], 2), "h2d_ms": round(st["h2d_ms"], 2),
            "compute_ms": round(compute, 2), "d2h_ms": round(st["d2h_ms"], 2),
            "parts_in_sequence_ms": round(st["h2d_ms"] + compute + st["d2h_ms"], 2),
            "h2d_gb": round(st["h2d_bytes"] / 1e9, 3), "d2h_gb": round(st["d2h_bytes"] / 1e9, 3),
            "h2d_gbs": round(st["h2d_bytes"] / max(st["h2d_ms"], 1e-9) / 1e6, 2),
            "d2h_gbs": round(st["d2h_bytes"] / max(st["d2h_ms"], 1e-9) / 1e6, 2),
            "h2d_overlapped_by_compute": overlap_fraction(ts, "h2d", "compute"),
            "compute_overlapped_by_copies": overlap_fraction(ts, "compute", "h2d"),
            "gflops_end_to_end": round(2 * st["products"] / wall / 1e9, 3),
            "device_peak_gb_measured": round(peak / 1e9, 3),
            "calls": 3, "warmup": 1}

    out["cfg5_streamed"] = dict(
        workload="cfg5 out-of-core aggregation: symmetric R-MAT n=68000000 deg 22 + self-loops (int64 row_ptr), "
                 "X 68000000x64 10% U(-1,1); A and X in pinned host memory, C to pinned host memory; "
                 "C sized by the exact bound min(N, P_i) (the default)",
        generation_s=round(gen, 2), **calls(B_.CBOUND_PRODUCTS))
    # the same calls planned with the row-pointer bound min(N, nnz(A_i) * max_k nnz(B_k)): no pass over
    # A's columns in the plan, about twice the pinned C reservation
    out["cfg5_streamed_rows_bound"] = dict(
        workload="the cfg5 out-of-core call above, C sized by the row-pointer bound", **calls(B_.CBOUND_ROWS))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--combine", type=int, default=0, metavar="F_OUT",
                    help="instead of the aggregation, time the combination step of the GCN layer "
                         "(Eq. 3): relu(C * W) with C the workload's aggregated features (computed once, "
                         "untimed) and a random dense W with F_OUT columns (aires_spmm)")
    ap.add_argument("--spmm-algo", default="auto", choices=["auto", "rows", "dense_tiles"],
                    help="kernel family of aires_spmm for --combine / --dense-h")
    ap.add_argument("--dense-h", type=int, default=0, metavar="F",
                    help="instead, time the next layer's aggregation A_norm * H with a dense H of F "
                         "columns (Eq. 1 with dense features; aires_spmm), A the workload's graph")
    ap.add_argument("--stream", action="store_true",
                    help="instead, the out-of-core schedule: A and X in pinned host memory, C back to "
                         "pinned host memory, one line per (feature width, budget)")
    ap.add_argument("--budget-gb", default="", help="--stream: comma-separated device budgets in GB (32)")
    ap.add_argument("--features", default="", help="--stream: comma-separated feature widths (the workload's)")
    ap.add_argument("--nodes", type=int, default=0, help="--stream: graph nodes (the workload's)")
    ap.add_argument("--max-tile-mb", type=int, default=0, help="--stream: cap on a tile's A bytes (0: none)")
    ap.add_argument("--storage", default="",
                    help="--stream: a directory; A's and X's arrays are written to files there; every call "
                         "reads X whole into HBM first, then A's tiles from their file (direct I/O) instead of "
                         "pinned memory (c_bound rows)")
    ap.add_argument("--segmentation", default="robw",
                    help="--stream: comma-separated segmentations of A: robw (row blocks, Algorithm 1) and/or "
                         "maxfill (segments filled to the slot, partial rows copied back, packed on the host "
                         "and sent again)")
    ap.add_argument("--c-on-device", action="store_true",
                    help="--stream: C stays in device memory instead of returning to pinned host memory")
    ap.add_argument("--c-bound", default="products", choices=["products", "rows"],
                    help="--stream: C bound of the plan, min(N, P_i) (a gather over A's columns) or "
                         "min(N, nnz(A_i) max_k nnz(B_k)) (row pointers only)")
    ap.add_argument("--sym-norm", action="store_true",
                    help="--stream: A's values derived on the device from its pattern (Eq. 2) instead of copied")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the extra records of the default run (cfg2 in core, cfg5 streamed)")
    ap.add_argument("--gather-probe-mib", type=int, default=0,
                    help="first run a random 4-byte gather from an array of this many MiB (sub-line reads of "
                         "known footprint for reading rocprofv3 FETCH_SIZE)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="first run one device copy of this many MiB (a known-size kernel for "
                         "scaling rocprofv3 FETCH_SIZE/WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU; --gpus %d is not supported "
              "(the path would shard by row blocks of A and C)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    import paper_2507_02006_amd as aires

    torch.cuda.set_device(0)
    if args.stream:
        return streamed(args)
    if args.workload not in WORKLOAD_NAMES:
        sys.exit("bench.py: workload %d is timed with --stream" % args.workload)
    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.gather_probe_mib:
        # a gather of known footprint: n random 4-byte reads from an array
        # of gather_probe_mib MiB (index_select), for reading the counters
        # of sub-line reads against the lines they touch
        n_src = args.gather_probe_mib << 18
        g = torch.Generator(device="cuda").manual_seed(23)
        src = torch.ones(n_src, dtype=torch.float32, device="cuda")
        idx = torch.randint(0, n_src, (n_src // 64,), generator=g, device="cuda")
        out = torch.index_select(src, 0, idx)
        torch.cuda.synchronize()
        ix = idx.cpu().numpy()
        print(json.dumps({"gather_probe": {"src_mib": args.gather_probe_mib, "reads": int(ix.size),
                                           "distinct_64B_lines": int(np.unique(ix // 16).size),
                                           "distinct_128B_lines": int(np.unique(ix // 32).size),
                                           "index_bytes": int(ix.size * 8), "out_bytes": int(ix.size * 4)}}),
              file=sys.stderr, flush=True)
        del src, idx, out
    t0 = time.perf_counter()
    A, B = workloads.workload(args.workload)
    gen_s = time.perf_counter() - t0
    dA, dB = aires.to_device(A), aires.to_device(B)
    if args.combine:
        return combine(args, A, B, dA, dB, gen_s)
    if args.dense_h:
        return dense_aggregate(args, A, dA, gen_s)
    torch.cuda.synchronize()
    run = in_core_run(A, B, dA, dB, args.steps, args.warmup)
    ms_per_step = run["ms_per_step"]
    P = run["P"]
    total_products = run["products"]
    roof = run["roofline"]
    roof["traffic"] = measured_traffic("cfg%d/numeric/%s" % (args.workload, run["dominant"]),
                                       roof["algorithmic_bytes"])
    # the counter bytes as a rate over this run's launch time, beside the
    # algorithmic (achieved) and gather-model rates
    roof["traffic_gbs"] = (round(roof["traffic"] / (roof["avg_launch_ms"] * 1e-3) / 1e9, 2)
                           if roof["traffic"] else None)
    res = {
        "metric": METRIC,
        "value": round(2 * total_products / (ms_per_step * 1e-3) / 1e9, 3),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "accumulation": "fp32 products; sums in 32-bit fixed point (at most 1e-6 rounding per entry) in "
                        "window rows whose bound allows it, fp32 elsewhere",
        "data": "synthetic (seeded R-MAT graph and uniform sparse features, generated on the host)",
        "config": {"workload": "cfg%d %s" % (args.workload, WORKLOAD_NAMES[args.workload]),
                   "m": A.nrows, "n": B.ncols, "nnz_a": A.nnz, "nnz_b": B.nnz,
                   "products": total_products, "nnz_c": run["nnz_c"], "tiles": run["tiles"],
                   "parallelism": "single GPU"},
        "roofline": {k: roof[k] for k in ("bound", "kernel", "achieved", "peak", "unit", "frac", "traffic",
                                          "algorithmic_bytes", "avg_launch_ms", "gather_model_gbs",
                                          "traffic_gbs")},
        "phases_ms": run["phases_ms"],
        "numeric_gflops": run["numeric_gflops"],
        "end_to_end_compulsory_gbs": run["end_to_end_compulsory_gbs"],
        "numeric_kind_ms": run["numeric_kind_ms"],
        "generation_s": round(gen_s, 2),
    }
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(A, B, P, args.cpu_seconds)
        model, ncpu = host_cpu()
        # a one-GPU share of the host: at most 16 threads
        allc = cpu_baseline(A, B, P, args.cpu_seconds / 2, threads=max(1, min(ncpu, 16)))
        allc["cpu_model"] = model
        res["cpu_baseline_all_cores"] = allc
    if args.workload == 3 and not args.no_extras:
        del dA, dB, A, B, P
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        res["extra_workloads"] = extras(args)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
