"""Benchmark: one EM iteration of the fused diagonal-GMM hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload large]

A step is one full EM iteration (E-step with statistic accumulation, then the
M-step) over the whole synthetic data set, already resident in HBM.  The
default workload is the paper-shape large one: N = 1e8 points, D = 128,
K = 1024 components (51.2 GB of fp32 data), random-point initialisation.

Prints one JSON line on stdout.  `roofline` covers the dominant kernel,
k_logz (log-densities of every point against every component, their
log-sum-exp, the exact refinement and log Z), timed over the timed steps with
the library's phase timer (HIP events recorded on the stream the kernels run
on).  Its algorithmic work is the log-density contraction over all N x K
pairs, 4*N*K*D flop per launch ([x | x^2] against [W | P], depth 2D), priced
against the peak of the MFMA type it runs on (bf16 for D <= 128 and D > 256,
where the fp32 operands are split in hi/lo bf16 parts and three products are
summed, fp32 in between).  The E-step as a whole is also reported against the 8*N*K*D
flop of the dense algorithm.  `cpu_baseline` times the fp64 CPU checker on a
bounded slice of the same data and scales it linearly in N (the E-step is
exactly linear in N).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
HBM_PEAK_GBS = 8000.0
METRIC = ("ms per EM iteration + % MFMA roofline (8\u00b7N\u00b7K\u00b7D flop/iter), "
          "N=1M..100M, K=1024, D=128")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def load_data(w, dev, chunk_rows=1 << 22):
    """Generates X chunk by chunk on the host (pinned buffers, generation of the next chunk
    overlapping the upload of the current one) and accumulates the column sums the
    random-point initialisation needs."""
    import numpy as np
    import torch
    import gmm_synth

    mix = gmm_synth.Mixture(w)
    x = torch.empty((w.n, w.d), dtype=torch.float32, device=dev)
    colsum = np.zeros(w.d)
    colsq = np.zeros(w.d)
    bufs = [torch.empty((min(chunk_rows, w.n), w.d), dtype=torch.float32, pin_memory=True)
            for _ in range(2)]
    starts = list(range(0, w.n, chunk_rows))
    results = {}
    nthreads = max(1, min(16, os.cpu_count() or 1))

    def gen(i):
        r0 = starts[i]
        r1 = min(w.n, r0 + chunk_rows)
        buf = bufs[i % 2][: r1 - r0]
        _, cs, cq = mix.rows(r0, r1, out=buf.numpy(), nthreads=nthreads, want_colstats=True)
        results[i] = (cs, cq)

    t0 = time.time()
    th = threading.Thread(target=gen, args=(0,))
    th.start()
    copy_done = [None, None]
    for i, r0 in enumerate(starts):
        th.join()
        r1 = min(w.n, r0 + chunk_rows)
        cs, cq = results.pop(i)
        colsum += cs
        colsq += cq
        x[r0:r1].copy_(bufs[i % 2][: r1 - r0], non_blocking=True)
        ev = torch.cuda.Event()
        ev.record()
        copy_done[i % 2] = ev
        if i + 1 < len(starts):
            nxt = (i + 1) % 2
            if copy_done[nxt] is not None:
                copy_done[nxt].synchronize()   # the buffer about to be refilled is uploaded
            th = threading.Thread(target=gen, args=(i + 1,))
            th.start()
        if i % 4 == 0 or i + 1 == len(starts):
            log(f"  data: {r1}/{w.n} rows ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    return x, mix, colsum, colsq


def gpu_clocks():
    """Current GPU clocks as rocm-smi reports them (None when it cannot be read)."""
    import subprocess
    try:
        out = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True,
                             text=True, timeout=20)
        info = json.loads(out.stdout)
        card = next(iter(info.values()))
        return {k: v for k, v in card.items() if "clock" in k.lower() and "sclk" in k.lower()
                or "mclk" in k.lower()} or None
    except Exception:
        return None


def cpu_model():
    """The host CPU's model name from /proc/cpuinfo (None when it cannot be read)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, mix, theta, sample_rows, iso=False):
    """The fp64 checker on the first `sample_rows` rows, one full EM iteration, scaled to N.
    It runs on ORACLE_THREADS host threads: the CPU share one GPU is given on the machines this
    is measured on (16), whatever the host's core count."""
    import oracle
    x = mix.rows(0, sample_rows, nthreads=max(1, min(16, os.cpu_count() or 1)))
    nthreads = oracle.default_threads()
    t0 = time.time()
    (oracle.iso_iterate if iso else oracle.iterate)(x, *theta, nthreads=nthreads)
    dt = time.time() - t0
    return {"value": dt * 1e3 * (w.n / sample_rows), "unit": "ms/iter", "cores": nthreads,
            "kind": "oracle", "host_cpus": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"one EM iteration (E-step, M-step, second sweep) over rows 0..{sample_rows} "
                      f"of the same data at Theta_0 on {nthreads} threads (the host's CPU share "
                      f"per GPU), {dt:.2f} s wall, scaled by N/{sample_rows}"}


COPY_BYTES = 2 << 30


def padded_d(d):
    """The library's padded dimension count (a multiple of 64 up to 256, of 128 above)."""
    return -(-d // 64) * 64 if d <= 256 else -(-d // 128) * 128


def calibrate_copy():
    """One device-to-device copy of COPY_BYTES: reads and writes exactly that many bytes, the
    scale for FETCH_SIZE / WRITE_SIZE."""
    import torch
    a = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES}), flush=True)


def source_digest():
    import hashlib
    src = os.path.join(ROOT, "paper_2606_10896_amd", "csrc", "flashgmm.hip")
    with open(src, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


ESTEP_KERNELS = ("k_prep_", "k_logz", "k_stats_", "k_sparse_", "k_reduce_")


def counter_per_call(csv_path, kernels=ESTEP_KERNELS, skip=0):
    """Sum of a rocprofv3 --pmc counter (KiB) over the dispatches whose kernel name contains one
    of `kernels`, per gmm_estep_accumulate call (a call starts with its k_prep_class dispatch),
    leaving out the first `skip` calls (the warm-up iterations): per E-step, or per k_logz
    launch when kernels = ("k_logz",)."""
    import csv
    with open(csv_path) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Dispatch_Id"]))
    tot, call, calls = 0.0, 0, set()
    for row in rows:
        name = row["Kernel_Name"]
        if ("copyBuffer" if "copyBuffer" in kernels else "k_prep_class") in name:
            call += 1
        if call > skip and any(k in name for k in kernels):
            tot += float(row["Counter_Value"])
            calls.add(call)
    return tot / max(len(calls), 1)


def write_traffic(workload, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, skip=2):
    """profiles/estep_traffic_<workload>.json from two counter runs of the bench (FETCH_SIZE,
    WRITE_SIZE; the first `skip` E-steps, the warm-up, left out) and the same counters over a
    COPY_BYTES device copy, which fix the scale of each counter."""
    f_copy = counter_per_call(copy_fetch_csv, ("copyBuffer",)) * 1024.0
    w_copy = counter_per_call(copy_write_csv, ("copyBuffer",)) * 1024.0
    f_scale, w_scale = COPY_BYTES / f_copy, COPY_BYTES / w_copy
    fetch = counter_per_call(fetch_csv, skip=skip) * 1024.0 * f_scale
    write = counter_per_call(write_csv, skip=skip) * 1024.0 * w_scale
    lf = counter_per_call(fetch_csv, ("k_logz",), skip) * 1024.0 * f_scale
    lw = counter_per_call(write_csv, ("k_logz",), skip) * 1024.0 * w_scale
    out = {"workload": workload, "bytes_per_call": fetch + write, "fetch_bytes": fetch,
           "write_bytes": write, "logz_bytes_per_launch": lf + lw, "logz_fetch_bytes": lf,
           "logz_write_bytes": lw, "fetch_scale": f_scale, "write_scale": w_scale,
           "warmup_calls_skipped": skip, "source_sha256": source_digest()}
    path = os.path.join(ROOT, "profiles", f"estep_traffic_{workload}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def measured_traffic(workload, key="logz_bytes_per_launch"):
    """HBM bytes per k_logz launch (or, with key="bytes_per_call", per E-step) from the
    committed counter runs (profiles/estep_traffic_<workload>.json), or None when the kernels
    have changed since."""
    path = os.path.join(ROOT, "profiles", f"estep_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha256") != source_digest():
        return None
    return t.get(key)


def bench_assign(args, w, x, th0, dev):
    """gmm_assign_topk with m = 2, tau = 1/K over all N points (the paper's multi-assignment,
    Sec. 4.3) at the parameters after the fit; timed with HIP events on the stream it runs on."""
    import numpy as np
    import torch
    import paper_2606_10896_amd as gmm
    k, d = w.k, w.d
    stream = torch.cuda.current_stream()
    wt, mu, var = (torch.from_numpy(a).to(dev) for a in th0)
    n_fit = w.iters if args.assign_fit < 0 else args.assign_fit
    if n_fit > 0:
        ws = gmm.workspace(w.n, d, k, device=dev)
        hist = torch.zeros(n_fit, dtype=torch.float64, device=dev)
        gmm.gmm_fit(x, wt, mu, var, n_fit, hist, ws, stream=stream)
        torch.cuda.synchronize()
        log(f"  fit: {n_fit} iterations, LL {hist[-1].item():.6e}")
        del ws
        torch.cuda.empty_cache()
    m, tau = 2, 1.0 / k
    wsa = gmm.workspace(w.n, d, k, m, device=dev)
    idx = torch.empty((w.n, m), dtype=torch.int32, device=dev)
    resp = torch.empty((w.n, m), dtype=torch.float32, device=dev)
    for _ in range(max(args.warmup, 1)):
        gmm.gmm_assign_topk(x, wt, mu, var, m, tau, idx, resp, wsa, stream=stream)
    torch.cuda.synchronize()
    steps = max(args.steps, 1)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        gmm.gmm_assign_topk(x, wt, mu, var, m, tau, idx, resp, wsa, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    kept2 = int((idx[:, 1] >= 0).sum().item())
    flop = 4.0 * w.n * k * d                  # log-densities of every (point, component) pair
    rate = flop / (ms * 1e-3) / 1e12
    # both passes screen on split-bf16 MFMA (three bf16 products per fp32 product) up to 128
    # and above 256 padded dimensions, on fp32 MFMA in between
    split = padded_d(d) <= 128 or padded_d(d) > 256
    peak = BF16_MFMA_PEAK_TFLOPS if split else FP32_MFMA_PEAK_TFLOPS
    how = "split-bf16 MFMA, bf16 peak" if split else "fp32 MFMA peak"
    print(json.dumps({
        "metric": "gmm_assign_topk time (m=2, tau=1/K)", "value": round(ms, 3), "unit": "ms",
        "higher_is_better": False, "n_gpus": 1, "steps": steps, "data": "synthetic",
        "config": {"workload": f"{w.name}: top-2 multi-assignment after {n_fit} EM iterations, "
                               f"N={w.n}, D={d}, K={k}", "n": w.n, "d": d, "k": k, "m": m,
                   "tau": tau},
        "second_rank_kept": kept2,
        "roofline": {"bound": "mfma", "kernel": "k_assign_theta + k_assign_collect (4*N*K*D flop "
                     f"of log-densities, {how}; both passes screen every pair)",
                     "achieved": round(rate, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(rate / peak, 4)}}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--kmeans", type=int, default=0, metavar="ITERS",
                    help="time only the k-means warm start (ITERS Lloyd iterations from the "
                         "random-point centres, then the hard mixture; one JSON line)")
    ap.add_argument("--kmeanspp", action="store_true",
                    help="time only the k-means++ seeding of the workload's K centres (one JSON "
                         "line, not the EM metric)")
    ap.add_argument("--assign", action="store_true",
                    help="time gmm_assign_topk (m = 2, tau = 1/K, Sec. 4.3) over all N points "
                         "after --assign-fit EM iterations from the initialisation (one JSON "
                         "line, not the EM metric)")
    ap.add_argument("--assign-fit", type=int, default=-1, metavar="ITERS",
                    help="EM iterations before the timed assignment (-1: the workload's own)")
    ap.add_argument("--rows", type=int, default=0,
                    help="take only the first ROWS rows of the workload (0 = all of them)")
    ap.add_argument("--ring-chunk", type=int, default=0,
                    help="out-of-core E-step from ordinary (pageable) host memory through a ring "
                         "of three page-locked chunks of RING_CHUNK rows "
                         "(gmm_estep_accumulate_ring; PCIe-inclusive, not the headline)")
    ap.add_argument("--stream-chunk", type=int, default=0,
                    help="rows per chunk of the out-of-core E-step (X in pinned host memory, "
                         "uploaded while the previous chunk runs); 0 = X resident in HBM "
                         "(the default and the reported value)")
    ap.add_argument("--covariance", choices=("diag", "iso"), default="diag",
                    help="diagonal components (default) or the paper's isotropic ones (one "
                         "variance per component, the *_iso calls)")
    ap.add_argument("--precision", choices=("exact", "screened"), default="exact",
                    help="exact E-step (default, the reported value) or the reduced-precision "
                         "one (gmm_estep_accumulate_screened: screened log-densities for every "
                         "pair, looser tolerances)")
    ap.add_argument("--from-init", type=int, default=-1, metavar="ITERS",
                    help="after the timed steps, also time ITERS iterations of one gmm_fit call "
                         "from the initialisation (-1: the workload's own iteration count, "
                         "0: skip)")
    ap.add_argument("--cpu-sample", type=int, default=1_000_000,
                    help="rows of the CPU-baseline slice (0 = skip)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only copy a 2 GiB device buffer once (the reference for the HBM byte "
                         "counters) and exit")
    ap.add_argument("--write-traffic", nargs=4, metavar="CSV",
                    help="write profiles/estep_traffic_<workload>.json from rocprofv3 counter "
                         "CSVs: bench FETCH_SIZE, bench WRITE_SIZE, copy FETCH_SIZE, copy "
                         "WRITE_SIZE (no GPU needed)")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(args.workload, *args.write_traffic)
        return
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported "
              "(the hot path is single-GPU; sharding is described, not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import gmm_synth
    import paper_2606_10896_amd as gmm

    gmm.load_library()
    w = gmm_synth.WORKLOADS[args.workload]
    if args.rows > 0:   # the first `rows` rows of the workload's data (same generator)
        import dataclasses
        w = dataclasses.replace(w, name=f"{w.name}[:{args.rows}]", n=args.rows)
    dev = torch.device("cuda:0")
    log(f"workload {w.name}: N={w.n} D={w.d} K={w.k}")
    x, mix, colsum, colsq = load_data(w, dev)
    if args.kmeanspp:
        u = torch.from_numpy(np.random.default_rng(w.init_seed).random(w.k)).to(dev)
        idx = torch.empty(w.k, dtype=torch.int64, device=dev)
        cen = torch.empty(w.k, w.d, dtype=torch.float32, device=dev)
        kws = torch.empty(gmm.load_library().gmm_kmeanspp_workspace_bytes(w.n), dtype=torch.uint8,
                          device=dev)
        gmm.gmm_kmeanspp(x, u, idx, cen, kws)   # warm-up
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        gmm.gmm_kmeanspp(x, u, idx, cen, kws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        print(json.dumps({"metric": "k-means++ seeding time", "value": round(ms, 3), "unit": "ms",
                          "higher_is_better": False, "n_gpus": 1, "data": "synthetic",
                          "config": {"workload": w.name, "n": w.n, "d": w.d, "k": w.k},
                          "ms_per_centre": round(ms / w.k, 4),
                          "x_gbs": round(4.0 * w.n * w.d * (w.k - 1) / (ms * 1e-3) / 1e9, 1)}),
              flush=True)
        return
    th0 = gmm_synth.random_point_init(w, mix, colsum, colsq)
    if args.kmeans > 0:
        wt, mu, var = (torch.from_numpy(a).to(dev) for a in th0)
        asg = torch.empty(w.n, dtype=torch.int32, device=dev)
        kws = gmm.workspace(w.n, w.d, w.k, 1, device=dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        gmm.gmm_kmeans(x, wt, mu, var, args.kmeans, asg, kws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        print(json.dumps({"metric": "k-means warm start time", "value": round(ms, 3),
                          "unit": "ms", "higher_is_better": False, "n_gpus": 1,
                          "data": "synthetic",
                          "config": {"workload": w.name, "n": w.n, "d": w.d, "k": w.k,
                                     "lloyd_iterations": args.kmeans},
                          "ms_per_assignment": round(ms / (args.kmeans + 1), 3)}), flush=True)
        return
    if args.assign:
        bench_assign(args, w, x, th0, dev)
        return
    iso = args.covariance == "iso"
    if iso:   # isotropic start: the mean over the dimensions of the init variances
        th0 = (th0[0], th0[1], th0[2].astype(np.float64).mean(1).astype(np.float32))
    wt, mu, var = (torch.from_numpy(a).to(dev) for a in th0)
    k, d = w.k, w.d
    nk = torch.zeros(k, dtype=torch.float64, device=dev)
    s = torch.zeros(k, d, dtype=torch.float64, device=dev)
    q = torch.zeros(k, d, dtype=torch.float64, device=dev)
    ll = torch.zeros(args.warmup + args.steps, dtype=torch.float64, device=dev)
    ws = gmm.workspace(w.n, d, k, device=dev)
    stream = torch.cuda.current_stream()

    if iso:
        q = torch.zeros(k, dtype=torch.float64, device=dev)
    screened = args.precision == "screened"
    if screened and iso:
        sys.exit("--precision screened runs the diagonal model only")
    estep = (gmm.gmm_estep_accumulate_iso if iso else
             gmm.gmm_estep_accumulate_screened if screened else gmm.gmm_estep_accumulate)
    mstep = gmm.gmm_mstep_iso if iso else gmm.gmm_mstep
    if args.stream_chunk > 0:
        if iso or screened:
            sys.exit("--stream-chunk runs the exact diagonal model only")
        # out-of-core: X in page-locked host memory, uploaded chunk by chunk
        rows = min(args.stream_chunk, w.n)
        xh = torch.empty((w.n, w.d), dtype=torch.float32, pin_memory=True)
        xh.copy_(x)
        del x
        torch.cuda.empty_cache()
        staging = torch.empty(2 * rows * w.d, dtype=torch.float32, device=dev)
        ws = gmm.workspace(rows, d, k, device=dev)
        copy_stream = torch.cuda.Stream()

        def estep(_x, *a, stream=None):
            gmm.gmm_estep_accumulate_streamed(xh, *a[:7], rows, staging, a[7], stream=stream,
                                              copy_stream=copy_stream)
        x = None
    if args.ring_chunk > 0:
        if iso or screened or args.stream_chunk > 0:
            sys.exit("--ring-chunk runs the exact diagonal model only")
        # out-of-core: X in ordinary host memory, through a ring of page-locked chunks
        rows = min(args.ring_chunk, w.n)
        xh = np.empty((w.n, w.d), dtype=np.float32)
        for r0 in range(0, w.n, 1 << 22):
            xh[r0:r0 + (1 << 22)] = x[r0:r0 + (1 << 22)].cpu().numpy()
        del x
        torch.cuda.empty_cache()
        ring = torch.empty((3, rows, w.d), dtype=torch.float32, pin_memory=True)
        staging = torch.empty(2 * rows * w.d, dtype=torch.float32, device=dev)
        ws = gmm.workspace(rows, d, k, device=dev)
        copy_stream = torch.cuda.Stream()

        def estep(_x, *a, stream=None):
            gmm.gmm_estep_accumulate_ring(xh, w.n, *a[:7], rows, ring, staging, a[7],
                                          stream=stream, copy_stream=copy_stream)
        x = None

    def step(i, ev=None):
        nk.zero_(); s.zero_(); q.zero_()
        if ev is not None:
            ev[0].record(stream)
        estep(x, wt, mu, var, nk, s, q, ll[i:i + 1], ws, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        mstep(nk, s, q, float(w.n), wt, mu, var, var_floor=1e-6, stream=stream)

    for i in range(args.warmup):
        step(i)
        torch.cuda.synchronize()
        log(f"  warmup step {i} done")
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    # the phase timer waits for each E-step call's last event, which would serialise the
    # chunks of an out-of-core call (no fill or upload overlapping the previous E-step)
    out_of_core = args.stream_chunk > 0 or args.ring_chunk > 0
    gmm.gmm_timing_enable(not out_of_core)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    phase_tot, ncalls = gmm.gmm_timing_read()
    gmm.gmm_timing_enable(False)
    phases = {p: round(v / max(ncalls, 1), 3) for p, v in phase_tot.items()}
    if out_of_core:
        phases = {p: None for p in phases}
    ms_step = (t1 - t0) * 1e3 / args.steps
    estep_ms = float(np.mean([a.elapsed_time(b) for a, b in events]))
    hist = ll.cpu().numpy()
    log(f"  loglik: {hist[0]:.6e} -> {hist[-1]:.6e}")
    log(f"  phases (ms per E-step): {phases}")
    flops = 8.0 * w.n * k * d
    dense_rate = flops / (estep_ms * 1e-3) / 1e12
    # dominant kernel: k_logz, its log-density contraction per launch: [x | x^2] against
    # [W | P] (depth 2D) for the diagonal model, 4 N K D flop; [x | ||x||^2] against
    # [mu / var | -1/(2 var)] (depth D + 1) for the isotropic one, 2 N K (D + 1) flop
    logz_ms = phases["logz"] or float("nan")
    # split-bf16 screening (three bf16 products per fp32 product) for D <= 128 and D > 256;
    # fp32 MFMA in between
    logz_b16 = padded_d(d) <= 128 or padded_d(d) > 256
    logz_peak = BF16_MFMA_PEAK_TFLOPS if logz_b16 else FP32_MFMA_PEAK_TFLOPS
    # the isotropic screening runs where the split-bf16 one does; in between the isotropic
    # calls take the diagonal kernel with tied variances
    iso_screen = iso and logz_b16
    logz_flop = 2.0 * w.n * k * (d + 1) if iso_screen else 4.0 * w.n * k * d
    logz_alg = logz_flop / (logz_ms * 1e-3) / 1e12
    dominant = max(phases, key=lambda p: phases[p] or 0.0)
    result = {
        "metric": METRIC,
        "value": round(ms_step, 3),
        "unit": "ms/iter",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("bf16 hi/lo split MFMA (screening log-densities), f32 MFMA (dense statistics), "
                  "f64 (exact pairs, sums)") if logz_b16 else
                 "f32 MFMA (log-densities, dense statistics), f64 (exact pairs, sums)",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {'isotropic' if iso else 'diag'}-GMM EM, N={w.n}, "
                               f"D={d}, K={k}, fp32 points from {w.k_true} seeded diagonal "
                               "Gaussians, random-point init",
                   "n": w.n, "d": d, "k": k, "parallelism": "single GPU",
                   "precision": ("screened: split-bf16 log-densities for every pair, no fp64 "
                                 "refinement" if screened else "exact")},
        "roofline": {"bound": "mfma",
                     "kernel": "k_logz (" + ("2*N*K*(D+1)" if iso_screen else "4*N*K*D")
                               + " flop of log-densities per launch, "
                               + ("bf16 MFMA peak; 3 bf16 products per fp32 product"
                                  if logz_b16 else "fp32 MFMA peak") + ")",
                     "achieved": round(logz_alg, 2), "peak": logz_peak, "unit": "TFLOP/s",
                     "frac": round(logz_alg / logz_peak, 4),
                     # counters were taken on the exact diagonal path's k_logz only
                     "traffic": None if (screened or iso) else measured_traffic(w.name),
                     "kernel_ms": logz_ms,
                     "executed_tflops": round(logz_alg * (3 if logz_b16 else 1), 2),
                     # k_logz reads X once: its X stream against the HBM peak
                     "x_stream_gbs": round(4.0 * w.n * d / (logz_ms * 1e-3) / 1e9, 1),
                     "dominant_phase": dominant, "phases_ms": phases,
                     "estep_ms": round(estep_ms, 3),
                     "estep_8nkd_tflops": round(dense_rate, 2),
                     "estep_8nkd_frac_fp32_peak": round(dense_rate / FP32_MFMA_PEAK_TFLOPS, 4),
                     "estep_8nkd_frac_bf16_peak": round(dense_rate / BF16_MFMA_PEAK_TFLOPS, 4)},
        "cpu_baseline": None,
    }
    if out_of_core:
        # no per-kernel figure: the chunks' kernels are not timed one by one here
        result["roofline"] = None
        result["x_upload_gbs"] = round(4.0 * w.n * d / (estep_ms * 1e-3) / 1e9, 1)
    if args.stream_chunk > 0:
        result["config"]["x_residency"] = (f"pinned host memory, uploaded in chunks of {rows} rows "
                                           "(PCIe-inclusive rate)")
    if args.ring_chunk > 0:
        result["config"]["x_residency"] = (f"pageable host memory, through a ring of three "
                                           f"page-locked chunks of {rows} rows (PCIe-inclusive "
                                           "rate)")
    n_init = w.iters if args.from_init < 0 else args.from_init
    if n_init > 0 and args.stream_chunk == 0 and args.ring_chunk == 0:
        # the whole trajectory from Theta_0 (the first iterations cost more than later ones)
        wt0, mu0, var0 = (torch.from_numpy(a).to(dev) for a in th0)
        hist = torch.zeros(n_init, dtype=torch.float64, device=dev)
        fit = (gmm.gmm_fit_iso if iso else gmm.gmm_fit_screened if screened else gmm.gmm_fit)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        fit(x, wt0, mu0, var0, n_init, hist, ws, var_floor=1e-6, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        tot = e0.elapsed_time(e1)
        result["from_init"] = {"iterations": n_init, "ms_total": round(tot, 2),
                               "ms_per_iter": round(tot / n_init, 3),
                               "note": "one gmm_fit call over iterations 0.." + str(n_init - 1)
                                       + " from the random-point initialisation"}
        log(f"  from init: {n_init} iterations in {tot:.1f} ms")
    result["gpu_clocks"] = gpu_clocks()
    if args.cpu_sample > 0:
        log("  cpu baseline ...")
        result["cpu_baseline"] = cpu_baseline(w, mix, th0, min(args.cpu_sample, w.n), iso)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
