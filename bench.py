"""Benchmark of the PIC hot path on one MI355X.

One step = the whole path on the 16-D blob workload (n = 50,000, d = 16,
10 Dirichlet(5)-sized blobs, sigma = median pair distance of a 1,000-point
sample): Gaussian affinity and degrees, W = D^-1 A written directly (dense
float32 W of 2.5e9 entries, 10 GB), v0, T = 50 power-iteration updates and
the exact 1-D k-means with k = 10.  Inputs are resident in HBM before the timed
region.

Prints one JSON line.  `value` is the power-iteration rate in GB/s of W
streamed (4 bytes per stored entry, 50 updates per step, divided by the
power-iteration time); `ms_per_step` is the end-to-end step.  The roofline
object is for the dominant kernel (the dense product), timed with HIP events
on the library's stream, and also as a fraction of the plain read stream
the device reaches over the same buffer in the same run (read_stream);
cpu_baseline is the float64 oracle on a bounded sample of the same workload
on the host cores (host described in cpu_baseline.host).

The same line carries the other workloads' figures under "workloads" (the
small dense blobs and rings, the fused operator on 64-D blobs, the CSR
path on the 2M-node kNN graph built on the GPU), each with its own
roofline object for its dominant kernel and its own oracle baseline;
--workload NAME prints one such workload as a line of its own.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP16_MFMA_PEAK_TFLOPS = 2500.0       # dense fp16 matrix cores, MI355X
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemv_traffic_blobs16d_n50000.json")
SYM_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sym_traffic_blobs16d_n50000.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def code_text(text: str) -> str:
    """C++ source with its comments removed and every run of whitespace
    made one space: what the compiler sees, so that an edit of a comment
    does not disown counter figures taken on the same kernel."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            out.append(" ")
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash(source: str = "gemv.hip") -> str:
    """Hash of a kernel source's code (comments and layout excluded)."""
    with open(os.path.join(ROOT, "paper_1604_02700_amd", "csrc", source)) as f:
        return hashlib.sha256(code_text(f.read()).encode()).hexdigest()[:16]


def measured_traffic(path: str = TRAFFIC_FILE, source: str = "gemv.hip",
                     key: str = "gemv_hip_sha"):
    """HBM bytes per product launch from the committed rocprofv3 counter
    runs, if they were taken on the current kernel source; else None."""
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get(key) != kernel_source_hash(source):
        return None
    return t.get("bytes_per_launch")


def host_info(threads_used: int) -> dict:
    """CPU model, sockets, physical cores and logical CPUs of this host, and
    the threads the oracle ran with."""
    model, sockets, cores = None, set(), set()
    phys = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k, v = k.strip(), v.strip()
                if k == "model name" and model is None:
                    model = v
                elif k == "physical id":
                    phys = v
                    sockets.add(v)
                elif k == "core id":
                    cores.add((phys, v))
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count()
    return {"cpu_model": model, "sockets": len(sockets) or None,
            "physical_cores": len(cores) or None, "logical_cpus": os.cpu_count(),
            "cpus_available_to_process": avail, "threads_used": threads_used}


def cpu_baseline(w, n_sample, T):
    """The oracle on the first n_sample points of the same workload."""
    import oracle
    X = w.X[:n_sample]
    t0 = time.perf_counter()
    W = oracle.affinity(X, w.sigma)
    W, deg, v0, _ = oracle.degree_normalize(W, copy=False)
    t1 = time.perf_counter()
    pi = oracle.power_iterate_dense(W, v0, "fixed", T)
    t2 = time.perf_counter()
    oracle.kmeans1d(pi.v, w.k)
    t3 = time.perf_counter()
    gbs = T * 4.0 * n_sample * n_sample / (t2 - t1) / 1e9
    return {"value": round(gbs, 3), "unit": "GB/s", "cores": oracle.num_threads(),
            "kind": "oracle", "host": host_info(oracle.num_threads()),
            "sample": (f"first {n_sample} of the {w.n} points" if n_sample < w.n
                       else f"the whole workload ({w.n} points)")
                      + f", dense W (float64 in the oracle, counted at 4 B/entry "
                        f"like the GPU), T = {T}, affinity to k-means",
            "e2e_s": round(t3 - t0, 3),
            "phases_s": {"affinity_normalise": round(t1 - t0, 3),
                         "power_iteration": round(t2 - t1, 3),
                         "kmeans": round(t3 - t2, 3)}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--n", type=int, default=50000)
    ap.add_argument("--T", type=int, default=50)
    ap.add_argument("--gemv-reps", type=int, default=20)
    ap.add_argument("--e2e-runs", type=int, default=10,
                    help="timed end-to-end runs (after one warm-up) for the median "
                         "and mean job times")
    ap.add_argument("--cpu-sample", type=int, default=50000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-converge", action="store_true")
    ap.add_argument("--no-sym", action="store_true",
                    help="skip the symmetric-storage figures of the headline line")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other workloads' figures of the headline line")
    ap.add_argument("--workload", default="blobs16d",
                    choices=["blobs16d", "blobs16d_sym", "blobs16d_host", "blobs64d", "knn8d",
                             "knn8d_random", "rings2d", "blobs2d", "moons", "circles3"],
                    help="blobs16d is the headline line; the others measure the "
                         "fused, CSR, small dense and cosine (the paper's "
                         "Experiment I shapes) paths")
    ap.add_argument("--wn", type=int, default=None,
                    help="points of a non-headline workload (its default if unset)")
    ap.add_argument("--copy-ref-gib", type=float, default=0.0,
                    help="also time a plain torch copy of this many GiB (the "
                         "reference kernel for counter scaling)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU "
              "path; N > 1 is not supported.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1604_02700_amd as g
    import workloads

    if args.workload == "blobs16d_sym":
        return sym_workload(args)
    if args.workload == "blobs16d_host":
        return host_workload(args)
    if args.workload != "blobs16d":
        return other_workload(args)

    dev = torch.device("cuda:0")
    tg0 = time.perf_counter()
    w = workloads.make("blobs16d", n=args.n if args.n != 50000 else None)
    gen_s = time.perf_counter() - tg0
    n, d, T, k = w.n, w.d, args.T, w.k
    log(f"bench: workload blobs16d n={n} d={d} sigma={float(w.sigma):.6g} T={T} k={k}")

    X = torch.from_numpy(w.X).to(dev)           # the first copy also starts the device
    torch.cuda.synchronize()
    h2d = []                                    # the host-to-device copy of X alone
    for _ in range(3):
        th0 = time.perf_counter()
        X.copy_(torch.from_numpy(w.X))
        torch.cuda.synchronize()
        h2d.append((time.perf_counter() - th0) * 1e3)
    h2d_ms = float(np.median(h2d))
    lda = g.padded_ld(n)
    A = torch.empty((n, lda), dtype=torch.float32, device=dev)
    v = torch.empty(n, dtype=torch.float64, device=dev)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    wbytes = 4.0 * n * n

    def step(record):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        ev[0].record(stream)
        ev[1].record(stream)
        W, deg, v0, nz = g.gpic_affinity_normalized(X, w.sigma, A)
        v.copy_(v0)
        ev[2].record(stream)
        pi = g.gpic_power_iterate_dense(W, v, None, "fixed", T, record_stats=False, n=n)
        ev[3].record(stream)
        km = g.gpic_kmeans1d(v, k)
        ev[4].record(stream)
        if record is not None:
            torch.cuda.synchronize()
            record.append([ev[i].elapsed_time(ev[i + 1]) for i in range(4)])
        return pi, km

    for i in range(args.warmup):
        step(None)
        log(f"bench: warmup step {i + 1}/{args.warmup} done")
    torch.cuda.synchronize()

    phases = []
    t0 = time.perf_counter()
    for i in range(args.steps):
        pi, km = step(phases)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log(f"bench: {args.steps} timed steps done in {wall:.3f} s")
    ph = np.array(phases)                     # ms per phase per step
    ms_step = wall * 1e3 / args.steps
    pi_ms = float(ph[:, 2].mean())
    value = T * wbytes / (pi_ms * 1e-3) / 1e9

    # the job from X resident on the device to labels on the device, run
    # by run (each ends with a synchronisation): median and mean
    runs = []
    for _ in range(args.e2e_runs):
        tr0 = time.perf_counter()
        step(None)
        torch.cuda.synchronize()
        runs.append(time.perf_counter() - tr0)
    e2e_fixed = {"runs": len(runs), "median_s": round(float(np.median(runs)), 5),
                 "mean_s": round(float(np.mean(runs)), 5)} if runs else None

    # dominant kernel: the dense product alone, on the same stream
    W = A
    y = torch.empty(n, dtype=torch.float64, device=dev)
    g.gpic_matvec_dense(W, v, y, n=n)
    # back-to-back launches between one event pair on the library's stream:
    # the average launch duration (events around every launch would add the
    # recording itself to each)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.gemv_reps):
        g.gpic_matvec_dense(W, v, y, n=n)
    ev1.record(stream)
    torch.cuda.synchronize()
    gemv_ms = ev0.elapsed_time(ev1) / args.gemv_reps
    alg_bytes = wbytes + 16.0 * n            # W once, v read, y written
    achieved = alg_bytes / (gemv_ms * 1e-3) / 1e9
    log(f"bench: product {gemv_ms:.4f} ms/launch, {achieved:.1f} GB/s")

    # the plain read stream over the same buffer: the read ceiling this
    # device reaches in the same run, timed like the product
    rs_n = W.numel() // 4 * 4
    sink = g.gpic_read_stream(W, rs_n)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.gemv_reps):
        g.gpic_read_stream(W, rs_n, sink)
    ev1.record(stream)
    torch.cuda.synchronize()
    rs_ms = ev0.elapsed_time(ev1) / args.gemv_reps
    rs_gbs = 4.0 * rs_n / (rs_ms * 1e-3) / 1e9
    read_stream = {"kernel": "read_stream_kernel", "bytes_per_launch": 4 * rs_n,
                   "avg_launch_ms": round(rs_ms, 5), "gbs": round(rs_gbs, 1),
                   "frac_of_peak": round(rs_gbs / HBM_PEAK_GBS, 4)}
    log(f"bench: read stream {rs_ms:.4f} ms/launch, {rs_gbs:.1f} GB/s")
    del sink

    conv = None
    if not args.no_converge:
        # one untimed run, then the median and mean of the timed runs
        out = g.pic_dense(X, w.sigma, k, "converge", 1000, w.eps, A=A)
        torch.cuda.synchronize()
        tcs = []
        for _ in range(max(args.e2e_runs, 1)):
            tc0 = time.perf_counter()
            out = g.pic_dense(X, w.sigma, k, "converge", 1000, w.eps, A=A)
            torch.cuda.synchronize()
            tcs.append(time.perf_counter() - tc0)
        tc = float(np.median(tcs))
        conv = {"e2e_s": round(tc, 5), "mean_s": round(float(np.mean(tcs)), 5),
                "iterations": out.pi.iterations, "converged": out.pi.converged,
                "eps": w.eps, "runs": len(tcs), "statistic": "median"}
        log(f"bench: to convergence {out.pi.iterations} updates, {tc:.4f} s")

    sym = None
    if not args.no_sym:
        # the same job with A stored once as its upper tiles (half the bytes
        # per update); a secondary figure, not the headline value
        r = measure_sym(g, w, X, T, k, args.steps, args.warmup, args.gemv_reps,
                        not args.no_converge)
        sym = {"e2e_fixed_T_s": round(r["ms_step"] / 1e3, 5),
               "ms_per_update": round(r["pi_ms"] / T, 5),
               "stored_bytes": r["stored_bytes"], "phases_ms": r["phases_ms"],
               "product_ms": round(r["prod_ms"], 5),
               "to_convergence": r["to_convergence"]}
        log(f"bench: symmetric storage {sym['e2e_fixed_T_s']} s per fixed-T job")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"bench: cpu baseline (oracle) on {args.cpu_sample} points ...")
        cpu = cpu_baseline(w, min(args.cpu_sample, n), T)
        log(f"bench: cpu baseline {cpu['value']} GB/s on {cpu['cores']} threads")

    copy_ref = None
    if args.copy_ref_gib > 0:
        m = int(args.copy_ref_gib * (1 << 30)) // 4
        src = torch.ones(m, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        for _ in range(5):
            dst.copy_(src)
        c1.record(stream)
        torch.cuda.synchronize()
        cms = c0.elapsed_time(c1) / 5
        copy_ref = {"bytes_read": 4 * m, "bytes_written": 4 * m,
                    "ms": round(cms, 5), "gbs_read_plus_write": round(8 * m / cms / 1e6, 1)}
        log(f"bench: copy reference {copy_ref}")
        del src, dst

    others = None
    if not args.no_workloads:
        # the other workloads' figures (bounded: a few steps each)
        others = {}
        for key, name, st, wu in (("blobs2d_c1", "blobs2d", 5, 2), ("rings2d_c2", "rings2d", 3, 1),
                                  ("fused_c4", "blobs64d", 2, 1), ("csr_c5", "knn8d", 3, 1)):
            log(f"bench: workload {name} ...")
            w2 = make_workload(name)
            others[key] = measure_path(g, torch, w2, st, wu, cpu=not args.no_cpu_baseline)
            log(f"bench: {name} e2e {others[key]['e2e_ms']} ms, "
                f"{others[key]['ms_per_update']} ms/update, roofline frac "
                f"{others[key]['roofline']['frac']}")
            del w2
            torch.cuda.empty_cache()

    traffic = measured_traffic()
    line = {
        "metric": "power-iteration GB/s of W streamed (% HBM peak); end-to-end "
                  "PIC seconds, n=50k",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": f"blobs16d: n={n}, d={d}, 10 Dirichlet(5) Gaussian "
                               f"blobs, sigma=median pair distance, dense float32 W, "
                               f"T={T} fixed updates, exact 1-D k-means k={k}",
                   "n": n, "d": d, "T": T, "k": k, "storage": "f32",
                   "accumulate": "f64", "parallelism": "single GPU"},
        "pct_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "e2e_fixed_T_s": round(ms_step / 1e3, 5),
        "e2e_fixed_T_runs": e2e_fixed,
        "excluded_from_e2e": {"generate_s": round(gen_s, 4), "h2d_X_ms": round(h2d_ms, 4),
                              "X_bytes": int(w.X.nbytes)},
        "phases_ms": {"affinity_degree_normalise_v0": round(float(ph[:, 1].mean()), 4),
                      "power_iteration": round(pi_ms, 4),
                      "kmeans": round(float(ph[:, 3].mean()), 4)},
        "to_convergence": conv,
        "roofline": {"bound": "hbm", "kernel": "gemv_kernel",
                     "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "avg_launch_ms": round(gemv_ms, 5),
                     "bytes_per_launch": alg_bytes,
                     "frac_of_read_stream": round(achieved / rs_gbs, 4)},
        "read_stream": read_stream,
        "symmetric_storage": sym,
        "cpu_baseline": cpu,
        "workloads": others,
    }
    if copy_ref is not None:
        line["copy_reference"] = copy_ref          # only in counter-scaling runs
    print(json.dumps(line), flush=True)


def measure_sym(g, w, X, T, k, steps, warmup, gemv_reps, converge):
    """The 16-D blobs job over the symmetric storage of A (packed upper tiles,
    2 n^2 bytes per product): the fixed-T pipeline timed over `steps`, the
    product alone, and (if asked) the to-convergence run, median of three
    after an untimed one."""
    import torch
    dev = X.device
    n = w.n
    As = torch.empty(g.sym_bytes(n) // 4, dtype=torch.float32, device=dev)
    v = torch.empty(n, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(record):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        As_, deg, v0, nz = g.gpic_affinity_sym(X, w.sigma, As)
        v.copy_(v0)
        ev[1].record(stream)
        g.gpic_power_iterate_sym(As, n, deg, v, None, "fixed", T, record_stats=False)
        ev[2].record(stream)
        g.gpic_kmeans1d(v, k)
        ev[3].record(stream)
        if record is not None:
            torch.cuda.synchronize()
            record.append([ev[i].elapsed_time(ev[i + 1]) for i in range(3)])
        return deg

    for _ in range(warmup):
        step(None)
    torch.cuda.synchronize()
    phases = []
    t0 = time.perf_counter()
    for _ in range(steps):
        deg = step(phases)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    ph = np.array(phases)
    pi_ms = float(ph[:, 1].mean())
    stored = float(g.sym_bytes(n))
    # the product alone on the library's stream: one event pair around all
    # the launches, so the host's per-call work (workspace, marshalling)
    # overlaps the device's
    y = torch.empty(n, dtype=torch.float64, device=dev)
    g.gpic_matvec_sym(As, n, deg, v, y)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(gemv_reps):
        g.gpic_matvec_sym(As, n, deg, v, y)
    b.record(stream)
    torch.cuda.synchronize()
    prod_ms = a.elapsed_time(b) / gemv_reps
    alg = stored + 24.0 * n                        # the stored tiles once, v, d, y
    conv = None
    if converge:
        out = g.pic_sym(X, w.sigma, k, "converge", 1000, w.eps, As=As)
        torch.cuda.synchronize()
        tcs = []
        for _ in range(3):
            tc0 = time.perf_counter()
            out = g.pic_sym(X, w.sigma, k, "converge", 1000, w.eps, As=As)
            torch.cuda.synchronize()
            tcs.append(time.perf_counter() - tc0)
        conv = {"e2e_s": round(float(np.median(tcs)), 5), "iterations": out.pi.iterations,
                "converged": out.pi.converged, "runs": 3, "statistic": "median"}
    del As
    return {"stored_bytes": stored, "ms_step": ms_step, "pi_ms": pi_ms,
            "phases_ms": {"affinity_sym_degree_v0": round(float(ph[:, 0].mean()), 4),
                          "power_iteration": round(pi_ms, 4),
                          "kmeans": round(float(ph[:, 2].mean()), 4)},
            "prod_ms": prod_ms, "alg_bytes": alg, "to_convergence": conv}


def sym_workload(args):
    """The headline workload (16-D blobs, n = 50,000, T = 50, k = 10) over the
    symmetric storage of A (packed upper tiles, 2 n^2 bytes per product):
    one JSON line, not the headline line."""
    import torch
    import paper_1604_02700_amd as g
    import workloads

    dev = torch.device("cuda:0")
    w = workloads.make("blobs16d", n=args.n if args.n != 50000 else None)
    n, T, k = w.n, args.T, w.k
    log(f"bench: workload blobs16d (symmetric storage) n={n} T={T}")
    X = torch.from_numpy(w.X).to(dev)
    r = measure_sym(g, w, X, T, k, args.steps, args.warmup, args.gemv_reps,
                    not args.no_converge)
    stored, pi_ms, prod_ms, alg = r["stored_bytes"], r["pi_ms"], r["prod_ms"], r["alg_bytes"]
    line = {"metric": "blobs16d over symmetric storage: power-iteration GB/s of stored "
                      "A streamed; end-to-end PIC seconds, n=50k",
            "value": round(T * stored / (pi_ms * 1e-3) / 1e9, 2), "unit": "GB/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(r["ms_step"], 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": DTYPE, "data": "synthetic",
            "config": {"workload": f"blobs16d: n={n}, d={w.d}, packed upper tiles of A "
                                   f"({stored / 1e9:.2f} GB), T={T}, k={k}", "n": n,
                       "storage": "f32 symmetric tiles", "accumulate": "f64"},
            "e2e_fixed_T_s": round(r["ms_step"] / 1e3, 5),
            "phases_ms": r["phases_ms"],
            "dense_equivalent_gbs": round(T * 4.0 * n * n / (pi_ms * 1e-3) / 1e9, 2),
            "to_convergence": r["to_convergence"],
            "roofline": {"bound": "hbm", "kernel": "sym_gemv_kernel + sym_finalize_kernel",
                         "achieved": round(alg / (prod_ms * 1e-3) / 1e9, 2),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(alg / (prod_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         "avg_launch_ms": round(prod_ms, 5), "bytes_per_launch": alg,
                         "traffic": measured_traffic(SYM_TRAFFIC_FILE, "sym.hip",
                                                     "sym_hip_sha")}}
    print(json.dumps(line), flush=True)


def host_workload(args):
    """The headline workload's dense W kept in pinned host memory and
    streamed to the device in row panels every update (the out-of-core
    path): a few fixed updates, one JSON line with the PCIe-inclusive rate."""
    import torch
    import paper_1604_02700_amd as g
    import workloads

    dev = torch.device("cuda:0")
    w = workloads.make("blobs16d", n=args.n if args.n != 50000 else None)
    n = w.n
    T = min(args.T, 3)
    log(f"bench: workload blobs16d, W in pinned host memory, n={n} T={T}")
    X = torch.from_numpy(w.X).to(dev)
    W, deg, v0, _ = g.gpic_affinity_normalized(X, w.sigma)
    Wh = torch.empty(W.shape, dtype=torch.float32, pin_memory=True)
    Wh.copy_(W)
    del W
    torch.cuda.synchronize()
    v = v0.clone()
    g.gpic_power_iterate_dense_host(Wh, v, None, "fixed", 1, record_stats=False, n=n)
    torch.cuda.synchronize()
    v.copy_(v0)
    t0 = time.perf_counter()
    g.gpic_power_iterate_dense_host(Wh, v, None, "fixed", T, record_stats=False, n=n)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    wbytes = 4.0 * n * n
    line = {"metric": "blobs16d with W in host memory: power-iteration GB/s of W streamed "
                      "over PCIe", "value": round(T * wbytes / t / 1e9, 2), "unit": "GB/s",
            "n_gpus": 1, "steps": T, "warmup": 1, "ms_per_step": round(t * 1e3 / T, 3),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": DTYPE,
            "data": "synthetic",
            "config": {"workload": f"blobs16d: n={n}, dense float32 W ({wbytes / 1e9:.1f} GB) "
                                   "in pinned host memory, two 64 MiB device panels",
                       "n": n, "T": T, "storage": "f32, host"},
            "note": "one step = one update; the W stream crosses PCIe every update"}
    print(json.dumps(line), flush=True)


# GPIC seconds the paper reports for its Experiment I shapes (Table 2:
# cosine similarity, at most 3 updates, eps = 1e-5/n, Tesla K40m)
PAPER_GPIC_S = {("moons", 15000): 3.99, ("circles3", 15000): 4.03,
                ("moons", 30000): 18.00, ("circles3", 30000): 18.03,
                ("moons", 45000): 45.07, ("circles3", 45000): 45.90}


DTYPE = "f32 storage, f64 arithmetic"
FUSED_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fused_traffic_blobs64d_n200000.json")
CSR_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "spmv_staged_traffic_knn8d_n2000000.json")


def _events(torch, stream, fn, reps):
    """Average time of `reps` back-to-back calls between one event pair on
    the library's stream (ms)."""
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    fn()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def knn8d_points(n=None):
    """The kNN workload's points (the generator alone: the graph is built
    on the GPU by the library)."""
    import workloads
    n = n or 2000000
    X, y = workloads.blobs_equal(n=n, d=8, k=50, seed=5)
    return workloads.Workload("knn8d", X, y, np.float32(1.0), 1e-5 / n, 50, "converge",
                              1000, "csr", 5)


def oracle_baseline(w, graph=None):
    """The oracle on a bounded sample of the same workload, in the unit of
    the GPU figure it stands beside."""
    import oracle
    th = oracle.num_threads()
    base = {"cores": th, "kind": "oracle", "host": host_info(th)}
    if w.path in ("dense", "cosine"):
        reps = 3 if w.n <= 10000 else 1          # the two small configurations
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            A = oracle.affinity(w.X, w.sigma) if w.path == "dense" else oracle.affinity_cosine(w.X)
            W, deg, v0, _ = oracle.degree_normalize(A, copy=False)
            t1 = time.perf_counter()
            pi = oracle.power_iterate_dense(W, v0, w.mode, w.max_iter, w.eps)
            t2 = time.perf_counter()
            oracle.kmeans1d(pi.v, w.k)
            t3 = time.perf_counter()
            ts.append((t1 - t0, t2 - t1, t3 - t2))
        ta, tp, tk = (float(np.median([t[i] for t in ts])) for i in range(3))
        return {**base, "value": round(pi.iterations * 4.0 * w.n * w.n / tp / 1e9, 3),
                "unit": "GB/s", "sample": f"the whole workload ({w.n} points, "
                f"{pi.iterations} updates), affinity to k-means"
                + (f", median of {reps} runs" if reps > 1 else ""),
                "e2e_s": round(ta + tp + tk, 4),
                "phases_s": {"affinity_normalise": round(ta, 4), "power_iteration": round(tp, 4),
                             "kmeans": round(tk, 4)}}
    if w.path == "fused":
        # one product's rows are independent: 1,000 evenly spaced rows,
        # scaled to the whole sweep
        m = 1000
        rows = (np.arange(m, dtype=np.int64) * w.n) // m
        v = np.full(w.n, 1.0 / w.n)
        t0 = time.perf_counter()
        oracle.matvec_onthefly_rows(w.X, w.sigma, np.ones(w.n), v, rows)
        t = (time.perf_counter() - t0) * w.n / m
        return {**base, "value": round(2.0 * w.n * w.n * w.d / t / 1e12, 5), "unit": "TFLOP/s",
                "sample": f"{m} evenly spaced rows of one on-the-fly product (every pair's "
                          f"affinity recomputed in float64), scaled by n / {m} to a sweep",
                "s_per_sweep_estimate": round(t, 3)}
    if w.path == "csr":
        rp, col, val = graph
        T = 5
        t0 = time.perf_counter()
        wn, deg, v0, _ = oracle.degree_normalize_csr(rp, col, val)
        t1 = time.perf_counter()
        oracle.power_iterate_csr(rp, col, wn, v0, "fixed", T)
        t2 = time.perf_counter()
        nnz = col.shape[0]
        b = 8.0 * nnz + 8.0 * (w.n + 1) + 16.0 * w.n
        return {**base, "value": round(T * b / (t2 - t1) / 1e9, 3), "unit": "GB/s",
                "sample": f"{T} updates of the power iteration over the whole graph "
                          f"({w.n} nodes, {nnz} entries), bytes counted as on the GPU",
                "s_per_update": round((t2 - t1) / T, 4), "normalise_s": round(t1 - t0, 4)}
    return None


def measure_path(g, torch, w, steps, warmup, cpu=True, graph_numbering="local"):
    """One workload through its path: end-to-end steps, the power-iteration
    loop alone, the dominant kernel against its roofline, and (optionally)
    the oracle beside it.  Returns a dict."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    X = torch.from_numpy(w.X).to(dev)
    T = w.max_iter
    info = {"workload": w.name, "n": w.n, "d": w.d, "path": w.path, "mode": w.mode,
            "T_or_cap": T, "k": w.k}
    graph = None
    if w.path == "csr":
        # the input graph built on the GPU (exact 32-NN, union, Gaussian
        # weights); "local": nodes numbered in the points' Morton order
        build = (lambda: g.gpic_knn_graph_local(X, 32, 1.0)) if graph_numbering == "local" \
            else (lambda: g.gpic_knn_graph(X, 32, 1.0) + (None,))
        build()
        torch.cuda.synchronize()
        tg = time.perf_counter()
        rp, col, val0, perm = build()
        torch.cuda.synchronize()
        info["graph_build_gpu_s"] = round(time.perf_counter() - tg, 4)
        info["graph_numbering"] = ("Morton order of the points" if graph_numbering == "local"
                                   else "the generator's point order")
        nnz = int(val0.numel())
        info["nnz"] = nnz
        graph = (rp, col, val0)

        def step():
            return g.pic_csr(rp, col, val0.clone(), w.k, w.mode, T, w.eps)
    elif w.path == "fused":
        def step():
            return g.pic_fused(X, w.sigma, w.k, w.mode, T, w.eps)
    elif w.path == "cosine":
        A = torch.empty((w.n, g.padded_ld(w.n)), dtype=torch.float32, device=dev)

        def step():
            return g.pic_cosine(X, w.k, w.mode, T, w.eps, W=A)
    else:
        A = torch.empty((w.n, g.padded_ld(w.n)), dtype=torch.float32, device=dev)

        def step():
            return g.pic_dense(X, w.sigma, w.k, w.mode, T, w.eps, A=A)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    times = []
    for _ in range(steps):
        t0 = time.perf_counter()
        out = step()
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    it = out.pi.iterations
    # the power-iteration loop alone, from the same start
    v = out.v0.clone()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    roof = {}
    if w.path == "csr":
        valn = val0.clone()
        valn, _, _, _ = g.gpic_degree_normalize_csr(rp, col, valn)
        e0.record(stream)
        g.gpic_power_iterate_csr(rp, col, valn, v, None, "fixed", it, record_stats=False)
        e1.record(stream)
        torch.cuda.synchronize()
        pi_ms = e0.elapsed_time(e1)
        bytes_it = 8.0 * nnz + 8.0 * (w.n + 1) + 16.0 * w.n
        rate = {"value": it * bytes_it / (pi_ms * 1e-3) / 1e9, "unit": "GB/s",
                "bytes_per_update": bytes_it}
        yv = torch.empty_like(v)
        kms = _events(torch, stream, lambda: g.gpic_matvec_csr(rp, col, valn, v, yv), 20)
        staged = nnz <= 64 * w.n
        kernel = ("spmv_staged_kernel" if staged else "spmv_kernel")
        traffic = measured_traffic(CSR_TRAFFIC_FILE, "power.hip", "power_hip_sha") \
            if (staged and graph_numbering == "local" and w.n == 2000000) else None
        roof = {"bound": "hbm", "kernel": kernel, "achieved": bytes_it / (kms * 1e-3) / 1e9,
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": traffic,
                "avg_launch_ms": kms, "bytes_per_launch": bytes_it}
        if graph_numbering != "local":
            roof["note"] = ("gpic_matvec_csr has no column-blocked copy: on a random "
                            "numbering the power iteration's blocked product is faster "
                            "than this kernel (ms_per_update)")
    elif w.path == "fused":
        e0.record(stream)
        g.gpic_power_iterate_fused(X, w.sigma, out.degree, v, None, "fixed", it,
                                   record_stats=False)
        e1.record(stream)
        torch.cuda.synchronize()
        pi_ms = e0.elapsed_time(e1)
        # algorithmic: the operator's 2 n^2 d flop per sweep (every ordered
        # pair), whatever the kernel evaluates; executed: up to 2^19 points
        # each pair once in row groups of G (group R covers the columns
        # from its own first row on), three fp16 part products per
        # coordinate, coordinates padded to 32-coordinate chunks
        flops = 2.0 * w.n * w.n * w.d
        G = 384 if w.d <= 64 else 256                 # rows per group of the symmetric product
        if w.n <= (1 << 19):
            groups = (w.n + G - 1) // G
            pairs = float(sum(G * (w.n - G * r) for r in range(groups)))
            kernel = "affinity_mfma_kernel (kApplySym) + fused_sym_reduce_kernel"
        else:
            pairs = float(w.n) * w.n
            kernel = "affinity_mfma_kernel (kApply)"
        exec_flops = 3 * 2.0 * pairs * 32 * ((w.d + 31) // 32)
        ms_upd = pi_ms / max(it, 1)
        rate = {"value": flops / (ms_upd * 1e-3) / 1e12, "unit": "TFLOP/s",
                "flops_per_sweep": flops}
        traffic = measured_traffic(FUSED_TRAFFIC_FILE, "affinity.hip", "affinity_hip_sha") \
            if w.n == 200000 else None
        roof = {"bound": "mfma", "kernel": kernel,
                "achieved": flops / (ms_upd * 1e-3) / 1e12,
                "peak": FP16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s", "traffic": traffic,
                "avg_launch_ms": ms_upd, "flops_per_launch": flops,
                "flops_note": "algorithmic 2 n^2 d per product (the Gram contraction of every "
                              "ordered pair) over the dense fp16 matrix-core peak (the Gram "
                              "runs on fp16 split operands); launch time = one update of the "
                              "loop (product + reduce + tau/update)",
                "pairs_evaluated_per_sweep": pairs,
                "fp16_mfma_flops_executed_per_sweep": exec_flops,
                "fp16_mfma_tflops_executed": round(exec_flops / (ms_upd * 1e-3) / 1e12, 2)}
    else:
        W = A
        e0.record(stream)
        g.gpic_power_iterate_dense(W, v, None, "fixed", it, record_stats=False, n=w.n)
        e1.record(stream)
        torch.cuda.synchronize()
        pi_ms = e0.elapsed_time(e1)
        bytes_it = 4.0 * w.n * w.n
        rate = {"value": it * bytes_it / (pi_ms * 1e-3) / 1e9, "unit": "GB/s",
                "bytes_per_update": bytes_it}
        yv = torch.empty(w.n, dtype=torch.float64, device=dev)
        kms = _events(torch, stream, lambda: g.gpic_matvec_dense(W, v, yv, n=w.n), 20)
        alg = bytes_it + 16.0 * w.n
        roof = {"bound": "hbm", "kernel": "gemv_kernel", "achieved": alg / (kms * 1e-3) / 1e9,
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "traffic": None, "avg_launch_ms": kms,
                "bytes_per_launch": alg}
    rate["value"] = round(rate["value"], 3)
    roof["achieved"] = round(roof["achieved"], 3)
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["avg_launch_ms"] = round(roof["avg_launch_ms"], 5)
    res = {"config": info, "steps": steps, "warmup": warmup,
           "e2e_ms": round(1e3 * float(np.median(times)), 4), "e2e_statistic": "median",
           "iterations": it, "converged": out.pi.converged, "pi_ms": round(pi_ms, 4),
           "ms_per_update": round(pi_ms / max(it, 1), 5), "rate": rate, "roofline": roof}
    paper = PAPER_GPIC_S.get((w.name, w.n))
    if paper is not None:
        # the paper's own GPIC time for this shape (another machine: context)
        res["paper_context"] = {"gpic_s": paper, "hardware": "Tesla K40m",
                                "source": "Table 2", "e2e_s_here": round(res["e2e_ms"] / 1e3, 5)}
    if cpu:
        host_graph = None
        if graph is not None:
            host_graph = tuple(t.cpu().numpy() for t in graph)
        log(f"bench: oracle baseline for {w.name} ...")
        res["cpu_baseline"] = oracle_baseline(w, host_graph)
    return res


def make_workload(name, n=None):
    import workloads
    if name in ("knn8d", "knn8d_random"):
        return knn8d_points(n)
    return workloads.make(name, n=n)


def other_workload(args):
    """One non-headline workload as a JSON line of its own."""
    import torch
    import paper_1604_02700_amd as g

    w = make_workload(args.workload, args.wn)
    log(f"bench: workload {args.workload} n={w.n} d={w.d} path={w.path} mode={w.mode}")
    copy_ref = None
    if args.copy_ref_gib > 0:
        # a plain copy of known size in the same process: the reference
        # that scales the HBM traffic counters of a profiling run
        dev = torch.device("cuda:0")
        m = int(args.copy_ref_gib * (1 << 30)) // 4
        src = torch.ones(m, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        copy_ref = {"bytes_read": 4 * m, "bytes_written": 4 * m, "copies": 3}
        del src, dst
        torch.cuda.empty_cache()
    r = measure_path(g, torch, w, args.steps, args.warmup, cpu=not args.no_cpu_baseline,
                     graph_numbering="random" if args.workload == "knn8d_random" else "local")
    line = {"metric": f"{args.workload}: power-iteration rate ({w.path} operator); "
                      f"end-to-end PIC seconds",
            "value": r["rate"]["value"], "unit": r["rate"]["unit"], "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": r["e2e_ms"],
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": DTYPE, "data": "synthetic", **r}
    if copy_ref is not None:
        line["copy_reference"] = copy_ref
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
