"""Benchmark of the vector-wise N:M SpMM hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload R2]
                    [--no-sweep] [--no-cpu-baseline]

A step is one call of nmspmm_run (the whole device path: gathered staging,
MFMA contraction, store) on the headline workload, m = n = k = 4096 fp32 at
16:32 (50 %) with V = 32.  Inputs are generated on the host, packed with
nmspmm_compress (offline, untimed) and resident in HBM before timing; the
timed launches rotate over enough copies of (A, Bc, idx, C) that no launch
finds its operands in L2 or the 256 MB Infinity Cache.

Prints ONE JSON line: the headline value (effective TFLOPS on useful flops
2 m n k N/M), the roofline of the kernel (per-launch HIP-event durations on
the launch stream), the CPU oracle timed on the host, a sweep over the other
workloads (75 / 87.5 % sparsity, the MLP shape, skinny decode shapes) and a
dense fp32 torch.matmul comparison.
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from nm_workloads import RUNS, make_run, table_runs  # noqa: E402

PEAK_FP32_TFLOPS = 157.3     # MI355X dense fp32 (vector = matrix), AMD spec
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, AMD spec
CACHE_BYTES = 288 << 20      # 256 MB Infinity Cache + 8 x 4 MB L2

# HBM traffic of the headline kernel from rocprofv3 --pmc FETCH_SIZE and
# WRITE_SIZE (KiB per dispatch), each scaled by the factor the same counter
# reads for a copy kernel of known size.  Keyed by workload, kernel variant
# and the hash of that variant's device sources: null once any differs.
TRAFFIC = {
    ("R2", "nm_tiled_kernel<128x512m32w16,bv1,ka32,nq4>,split1", "ea2de4c5dc081452"): {
        "fetch_kib": 165179.4, "fetch_factor": 1.99995,
        "write_kib": 65536.0, "write_factor": 1.00000,
    },
}


def traffic_bytes(entry):
    """Calibrated read + write bytes per launch from one TRAFFIC entry."""
    return 1024.0 * (entry["fetch_kib"] * entry["fetch_factor"] + entry["write_kib"] * entry["write_factor"])


def kernel_source_sha(kernel_name):
    """Hash of the device sources of the named kernel variant: the tiled
    kernel's header plus its tile's instantiation unit, or the streaming
    kernel's file (a change invalidates TRAFFIC)."""
    csrc = os.path.join(ROOT, "paper_2503_01253_amd", "csrc")
    files = ["nmspmm_tiled.h"]
    if kernel_name.startswith("nm_tiled_kernel<"):
        files.append(f"nmspmm_tiled_{kernel_name.split('<')[1].split(',')[0]}.hip")
    elif kernel_name.startswith("nm_skinny_kernel<"):
        files.append("nmspmm_skinny.hip")
    elif kernel_name.startswith("nm_stream_kernel<"):
        files.append("nmspmm_stream.hip")
    elif kernel_name.startswith("nm_gather_kernel<"):
        files.append("nmspmm_gather.hip")
    elif kernel_name.startswith("nm_rowgather_kernel<"):
        files.append("nmspmm_rowgather.hip")
    else:
        files.append("nmspmm_kernels.hip")
    h = hashlib.sha256()
    for name in files:
        h.update(name.encode())
        h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class Workload:
    """Device-resident copies of one run's operands, rotated across launches."""

    def __init__(self, run, torch, nm, min_copies=1, with_dense=False):
        self.run = run
        self.torch = torch
        self.nm = nm
        A, Bp, _ = make_run(run)
        Bc, idx = nm.nmspmm_compress(Bp, run.N, run.M, run.V)
        per_copy = A.nbytes + Bc.nbytes + idx.nbytes + 4 * run.m * run.n
        self.copies = max(min_copies, int(np.ceil(2 * CACHE_BYTES / per_copy)))
        dev = torch.device("cuda")
        tA, tBc, tidx = (torch.from_numpy(x).to(dev) for x in (A, Bc, idx))
        self.sets = []
        for c in range(self.copies):
            self.sets.append((tA if c == 0 else tA.clone(), tBc if c == 0 else tBc.clone(),
                              tidx if c == 0 else tidx.clone(),
                              torch.empty((run.m, run.n), dtype=torch.float32, device=dev)))
        self.ptrs = [(a.data_ptr(), b.data_ptr(), i.data_ptr(), c.data_ptr()) for a, b, i, c in self.sets]
        # split-k through a workspace where the kernel takes one (launches on
        # one stream run one at a time, so one workspace serves every copy)
        need = nm.nmspmm_workspace_bytes(run.m, run.n, run.k, run.N, run.M, run.V)
        self.ws = torch.empty(need, dtype=torch.uint8, device=dev) if need > 0 else None
        self.dense = None
        if with_dense:
            tB = torch.from_numpy(Bp).to(dev)
            self.dense = [(s[0], tB if c == 0 else tB.clone(), torch.empty_like(s[3]))
                          for c, s in enumerate(self.sets)]
        self.host_A, self.host_Bp = A, Bp

    def launch(self, i, stream_handle):
        r = self.run
        a, b, x, c = self.ptrs[i % self.copies]
        if self.ws is None:
            st = self.nm.nmspmm_run_ptr(a, b, x, c, r.m, r.n, r.k, r.N, r.M, r.V, stream_handle)
        else:
            st = self.nm.lib().nmspmm_run_ws(a, b, x, c, r.m, r.n, r.k, r.N, r.M, r.V, ctypes.c_float(1.0),
                                             None, 0, self.ws.data_ptr(), self.ws.numel(), stream_handle)
        if st != 0:
            raise RuntimeError(f"nmspmm_run failed: {self.nm.nmspmm_status_string(st)}")

    def kernel_label(self):
        """The kernel variant's name, as launched: with the workspace when the
        shape takes one."""
        r = self.run
        if self.ws is not None:
            return self.nm.nmspmm_kernel_name_ws(r.m, r.n, r.k, r.N, r.M, r.V)
        return self.nm.nmspmm_kernel_name(r.m, r.n, r.k, r.N, r.M, r.V)

    def launch_dense(self, i):
        a, b, c = self.dense[i % self.copies]
        self.torch.matmul(a, b, out=c)

    def free(self):
        self.sets = None
        self.dense = None
        self.ws = None


def warm_gpu(torch, fn, seconds):
    """Launch `fn` until `seconds` of wall time have passed.  A cold MI355X
    runs the first tens of milliseconds of work ~10 % slower (clock ramp), so
    every timed batch is preceded by this much back-to-back work."""
    t = time.perf_counter()
    i = 0
    while time.perf_counter() - t < seconds:
        for _ in range(8):
            fn(i)
            i += 1
        torch.cuda.synchronize()


def time_launches(torch, fn, steps, warmup, warm_seconds=0.0):
    """Warm up (`warmup` launches, after at least `warm_seconds` of work),
    then time `steps` launches: total wall (events around the whole batch)
    and per-launch durations (an event pair around each launch, on the
    stream the kernel runs on)."""
    stream = torch.cuda.current_stream()
    if warm_seconds > 0:
        warm_gpu(torch, fn, warm_seconds)
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(steps):
        starts[i].record(stream)
        fn(warmup + i)
        ends[i].record(stream)
    t1.record(stream)
    torch.cuda.synchronize()
    per = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return t0.elapsed_time(t1), per


def pct(xs, q):
    xs = sorted(xs)
    return xs[min(len(xs) - 1, max(0, int(round(q * (len(xs) - 1)))))]


def time_graph(torch, launch, copies, batches, reps):
    """Per-launch time from replays of a HIP graph that holds one launch per
    operand copy (no host launch overhead between kernels): `batches` timed
    batches of `reps` replays each; returns per-launch ms for every batch."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(min(3, copies)):
            launch(i, s.cuda_stream)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        h = torch.cuda.current_stream().cuda_stream
        for i in range(copies):
            launch(i, h)
    warm_gpu(torch, lambda i: g.replay(), 0.2)
    out = []
    for _ in range(batches):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) / (reps * copies))
    del g
    return out


def cpu_baseline(run, A, Bp, target_s, threads=None):
    """The fp64 CPU oracle on the same workload, timed on the host cores
    (`threads` OpenMP threads; default: all)."""
    import oracle
    Bc, idx = oracle.compress(Bp, run.N, run.M, run.V)
    all_threads = oracle.max_threads()
    threads = threads or all_threads
    oracle.set_threads(threads)
    # calibrate on a few rows, then pick a row sample worth about target_s
    rows = min(run.m, 16)
    t = time.perf_counter()
    oracle.spmm(A[:rows], Bc, idx, rows, run.n, run.k, run.N, run.M, run.V)
    per_row = max(time.perf_counter() - t, 1e-6) / rows
    rows = int(min(run.m, max(1, target_s / per_row)))
    reps = max(1, int(target_s / (per_row * rows)))
    As = np.ascontiguousarray(A[:rows])
    times = []
    for _ in range(reps):
        t = time.perf_counter()
        oracle.spmm(As, Bc, idx, rows, run.n, run.k, run.N, run.M, run.V)
        times.append(time.perf_counter() - t)
    oracle.set_threads(all_threads)
    dt = statistics.median(times)
    flops = 2.0 * rows * run.n * run.w
    return {
        "value": flops / dt / 1e12, "unit": "TFLOPS", "cores": threads, "kind": "oracle",
        "sample": (f"{run.name}: {rows} of {run.m} rows of A (full k, n), fp64 oracle, "
                   f"median of {reps} run(s), {dt:.2f} s each"),
    }


def measured_roofs(torch):
    """The two roofs as this GPU reaches them, from bench/micro's kernels: a
    streaming read of 4 GiB (well past the 256 MB Infinity Cache) and an
    fp32 MFMA loop of independent v_mfma_f32_32x32x2_f32 chains.  Best of
    several launch shapes, median of the timed launches of each."""
    path = os.path.join(ROOT, "bench", "micro", "libnm_micro.so")
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built: run `python bench/micro/build.py`")
    L = ctypes.CDLL(path)
    L.nm_micro_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    L.nm_micro_mfma_f32.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    L.nm_micro_mfma_f32_flops.argtypes = [ctypes.c_int, ctypes.c_int]
    L.nm_micro_mfma_f32_flops.restype = ctypes.c_double
    h = torch.cuda.current_stream().cuda_stream
    nbytes = 4 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    hbm = {}
    for blocks in (1024, 2048, 4096, 8192):
        sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")

        def rd(i, blocks=blocks, sink=sink):
            if L.nm_micro_hbm_read(buf.data_ptr(), nbytes, sink.data_ptr(), blocks, h) != 0:
                raise RuntimeError("nm_micro_hbm_read failed")
        _, per = time_launches(torch, rd, 10, 2, 0.1)
        hbm[blocks] = nbytes / (statistics.median(per) * 1e-3) / 1e9
    del buf
    # the floor of the memory-bound decode run: one streaming read of R5a's
    # algorithmic bytes, launch and ramp included (graph replay over copies
    # past the Infinity Cache), best of 256-1024 workgroups
    r5a = RUNS["R5a"]
    small = int(r5a.alg_bytes) // 256 * 256
    copies = max(4, int(600e6 // small))
    bufs = [torch.ones(small // 4, dtype=torch.float32, device="cuda") for _ in range(copies)]
    floor = {}
    for blocks in (256, 512, 1024):
        sink = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")

        def rd_small(i, hs, blocks=blocks, sink=sink):
            if L.nm_micro_hbm_read(bufs[i].data_ptr(), small, sink.data_ptr(), blocks, hs) != 0:
                raise RuntimeError("nm_micro_hbm_read failed")
        floor[blocks] = statistics.median(time_graph(torch, rd_small, copies, 5, max(1, 400 // copies)))
    del bufs
    best_small = min(floor, key=floor.get)
    mfma = {}
    iters = 2048
    for blocks in (256, 512, 1024, 2048):
        sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

        def mm(i, blocks=blocks, sink=sink):
            if L.nm_micro_mfma_f32(sink.data_ptr(), iters, blocks, h) != 0:
                raise RuntimeError("nm_micro_mfma_f32 failed")
        _, per = time_launches(torch, mm, 10, 2, 0.1)
        mfma[blocks] = L.nm_micro_mfma_f32_flops(iters, blocks) / (statistics.median(per) * 1e-3) / 1e12
    torch.cuda.empty_cache()
    best_hbm, best_mfma = max(hbm, key=hbm.get), max(mfma, key=mfma.get)
    return {
        "hbm_read_gbs": round(hbm[best_hbm], 1), "hbm_read_blocks": best_hbm,
        "mfma_f32_tflops": round(mfma[best_mfma], 2), "mfma_f32_blocks": best_mfma,
        "r5a_read_floor_us": round(floor[best_small] * 1e3, 2), "r5a_read_floor_bytes": small,
        "r5a_read_floor_blocks": best_small,
        "spec_hbm_gbs": PEAK_HBM_GBS, "spec_fp32_tflops": PEAK_FP32_TFLOPS,
        "source": "bench/micro/nm_micro.hip (4 GiB streaming read; 8 chains of v_mfma_f32_32x32x2_f32 per wave; "
                  "the R5a floor: one read of its algorithmic bytes per graph-replayed launch)",
    }


def measure(torch, nm, run, steps, warmup, with_dense, graph=False, warm_seconds=0.2):
    """Time one workload.  Per-launch HIP events on the launch stream for
    launches long enough that host overhead hides behind them; for the
    microsecond-scale ones (graph=True) replays of a captured HIP graph, so
    the figure is the kernels' own time.  Reports median, p10 and p90."""
    w = Workload(run, torch, nm, with_dense=with_dense)
    handle = torch.cuda.current_stream().cuda_stream
    total_ms, per = time_launches(torch, lambda i: w.launch(i, handle), steps, warmup, warm_seconds)
    res = {
        "workload": run.name, "m": run.m, "n": run.n, "k": run.k, "N": run.N, "M": run.M,
        "V": run.V, "kernel": w.kernel_label(),
        "copies": w.copies, "ms_per_step": total_ms / steps,
        "kernel_ms_mean": statistics.fmean(per), "timing": "per-launch events",
    }
    if graph:
        per = time_graph(torch, w.launch, w.copies, 7, max(1, 200 // w.copies))
        res["timing"] = "graph replay"
        res["kernel_ms_mean"] = statistics.fmean(per)
    res["kernel_ms_median"] = statistics.median(per)
    res["kernel_ms_p10"] = pct(per, 0.1)
    res["kernel_ms_p90"] = pct(per, 0.9)
    res["eff_tflops"] = run.useful_flops / (res["kernel_ms_median"] * 1e-3) / 1e12
    res["hbm_gbs_alg"] = run.alg_bytes / (res["kernel_ms_median"] * 1e-3) / 1e9
    ai = run.useful_flops / run.alg_bytes
    roof = min(PEAK_FP32_TFLOPS, ai * PEAK_HBM_GBS / 1e3)
    res["roof_tflops"] = roof
    res["roof_frac"] = res["eff_tflops"] / roof
    res["bound"] = "hbm" if ai * PEAK_HBM_GBS / 1e3 < PEAK_FP32_TFLOPS else "mfma"
    if with_dense:
        if graph:
            d_per = time_graph(torch, lambda i, h: w.launch_dense(i), w.copies, 5,
                               max(1, 100 // w.copies))
        else:
            _, d_per = time_launches(torch, lambda i: w.launch_dense(i), max(10, steps // 4), 3, 0.2)
        d_ms = statistics.median(d_per)
        res["dense_matmul_ms"] = d_ms
        res["speedup_vs_dense"] = d_ms / res["kernel_ms_median"]
        res["ideal_speedup"] = run.M / run.N
    w.free()
    return res, w


def measure_extras(torch, nm):
    """The steps beside the product: the fused epilogue of nmspmm_run_ex on the
    MLP-shaped run (alpha = M/N, bias, GELU, against the plain product), the
    device packer nmspmm_compress_device on the headline's dense B, and Eq. 2's
    confusion matrix nmspmm_confusion on the headline's output size."""
    out = {}
    r = RUNS["R4"]
    w = Workload(r, torch, nm, min_copies=2)
    bias = torch.randn(r.n, device="cuda")
    h = torch.cuda.current_stream().cuda_stream
    L = nm.lib()

    def ex(i):
        a, b, x, c = w.ptrs[i % w.copies]
        st = L.nmspmm_run_ex(a, b, x, c, r.m, r.n, r.k, r.N, r.M, r.V, float(r.M / r.N),
                             bias.data_ptr(), nm.NMSPMM_ACT_GELU, h)
        if st != 0:
            raise RuntimeError(nm.nmspmm_status_string(st))
    _, plain = time_launches(torch, lambda i: w.launch(i, h), 20, 3, 0.2)
    _, fused = time_launches(torch, ex, 20, 3, 0.2)
    out["epilogue"] = {
        "workload": r.describe(), "epilogue": "gelu(M/N * C + bias)",
        "kernel": nm.nmspmm_kernel_name(r.m, r.n, r.k, r.N, r.M, r.V),
        "plain_ms": statistics.median(plain), "fused_ms": statistics.median(fused),
    }
    w.free()
    del bias
    r = RUNS["R2"]
    A, Bp, _ = make_run(r)
    dB = torch.from_numpy(Bp).cuda()
    wr = (r.k // r.M) * r.N
    dBc = torch.empty((wr, r.n), dtype=torch.float32, device="cuda")
    didx = torch.empty((wr, r.n // r.V), dtype=torch.uint8, device="cuda")
    _, per = time_launches(torch, lambda i: nm.nmspmm_compress_device(dB, dBc, didx, r.N, r.M, r.V),
                           20, 3, 0.2)
    ms = statistics.median(per)
    moved = 4.0 * r.k * r.n + 4.0 * wr * r.n + wr * (r.n // r.V)
    out["device_compress"] = {"workload": f"B of {r.name}: {r.k} x {r.n}, {r.N}:{r.M}, V={r.V}",
                              "ms": ms, "gb_s": moved / (ms * 1e-3) / 1e9}
    del dB, dBc, didx
    torch.cuda.empty_cache()
    # Eq. 2's confusion matrix on the headline's m x n output: two reads and
    # one write of 4 bytes per output, over two sets of arrays (384 MB, past
    # the Infinity Cache)
    sets = [[torch.randn(r.m, r.n, device="cuda") for _ in range(3)] for _ in range(2)]

    def cf(i):
        cs, cd, wt = sets[i % 2]
        st = L.nmspmm_confusion(cs.data_ptr(), cd.data_ptr(), wt.data_ptr(), r.m, r.n, h)
        if st != 0:
            raise RuntimeError(nm.nmspmm_status_string(st))
    _, per = time_launches(torch, cf, 40, 4, 0.2)
    ms = statistics.median(per)
    moved = 12.0 * r.m * r.n
    out["eq2_confusion"] = {"workload": f"W = |C' - C| / (m*n) on {r.m} x {r.n} fp32 outputs",
                            "ms": ms, "gb_s": moved / (ms * 1e-3) / 1e9,
                            "frac_hbm_peak": moved / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    del sets
    torch.cuda.empty_cache()
    # decode batches of 1, 2 and 4 rows on the skinny shape (the row-gather
    # kernel: one launch, A gathered from L2), graph replay; HBM-bound
    dec = []
    for mm in (1, 2, 4):
        rr = dataclasses.replace(RUNS["R5a"], name=f"R5a@m={mm}", m=mm)
        res, _ = measure(torch, nm, rr, 20, 3, False, graph=True)
        gbs = rr.alg_bytes / (res["kernel_ms_median"] * 1e-3) / 1e9
        dec.append({"m": mm, "kernel": res["kernel"], "us": round(res["kernel_ms_median"] * 1e3, 2),
                    "alg_gb_s": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 3)})
        torch.cuda.empty_cache()
    out["decode_batches"] = {"workload": "m x 8192 x 8192 (m x n x k), 4:32, V=64, normal seed=1008", "runs": dec}
    out["plain_call"] = plain_call(torch, nm)
    return out


def time_batch(torch, fn, steps, warmup):
    """Whole-batch time per call of `steps` back-to-back launches (events
    around the batch only, so nothing is enqueued between the calls)."""
    warm_gpu(torch, fn, 0.2)
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        fn(warmup + i)
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def plain_call(torch, nm):
    """nmspmm_run as a caller without a workspace makes it on the short
    products (the direct-gather kernel with the workspace the library caches
    for the stream), against nmspmm_run_ws with a caller workspace and against
    the kernels that take none: eager launches from Python, back to back."""
    L = nm.lib()
    h = torch.cuda.current_stream().cuda_stream
    rows = []
    for name in ("R5b", "R5c"):
        r = RUNS[name]
        w = Workload(r, torch, nm, min_copies=2)

        def plain(i, w=w, r=r):
            a, b, x, c = w.ptrs[i % w.copies]
            if L.nmspmm_run(a, b, x, c, r.m, r.n, r.k, r.N, r.M, r.V, h) != 0:
                raise RuntimeError("nmspmm_run failed")

        def none(i, w=w, r=r):
            a, b, x, c = w.ptrs[i % w.copies]
            if L.nmspmm_run_tuned(a, b, x, c, r.m, r.n, r.k, r.N, r.M, r.V, ctypes.c_float(1.0), None, 0,
                                  None, 0, None, h) != 0:
                raise RuntimeError("nmspmm_run_tuned failed")

        us = {lab: round(1e3 * statistics.median(time_batch(torch, fn, 400, 20) for _ in range(3)), 2)
              for lab, fn in (("nmspmm_run_us", plain), ("nmspmm_run_ws_us", lambda i, w=w: w.launch(i, h)),
                              ("no_workspace_us", none))}
        rows.append({"workload": name, "kernel": nm.nmspmm_kernel_name(r.m, r.n, r.k, r.N, r.M, r.V),
                     "kernel_no_workspace":
                         L.nmspmm_kernel_name_tuned(r.m, r.n, r.k, r.N, r.M, r.V, 0, None).decode(),
                     **us})
        w.free()
        torch.cuda.empty_cache()
    return {"timing": "400 back-to-back eager launches from Python, whole-batch time per call, median of 3",
            "runs": rows}


def summary_row(res, roofs):
    """One workload's compact record: kernel, time, effective rate, fraction
    of its roof (spec and, where measured, the measured roof), speedup over
    the dense fp32 GEMM and the ideal M/N."""
    run = RUNS.get(res["workload"]) or table_runs()[res["workload"]]
    frac_meas = None
    if roofs:
        ai = run.useful_flops / run.alg_bytes
        roof = min(roofs["mfma_f32_tflops"], ai * roofs["hbm_read_gbs"] / 1e3)
        frac_meas = round(res["eff_tflops"] / roof, 3)
    return [run.name, res["kernel"], round(res["kernel_ms_median"] * 1e3, 2), round(res["eff_tflops"], 1),
            round(res["roof_frac"], 3), res["bound"], frac_meas, round(res.get("speedup_vs_dense", 0.0), 2),
            run.M / run.N]


def device_clocks():
    """Current clocks as rocm-smi reports them (None where it is unavailable)."""
    import subprocess
    try:
        out = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True,
                             timeout=20).stdout
    except (OSError, subprocess.SubprocessError):
        return None
    lines = [ln.strip() for ln in out.splitlines() if "clk" in ln.lower() and "Mhz" in ln]
    return lines[:8] or None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="R2", choices=sorted(RUNS) + sorted(table_runs()),
                    help="the headline run (default R2), another benchmark run, or a point of the shape x "
                         "sparsity sweep (A-32 .. F-4), e.g. for counter passes with --launches-only")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-table", action="store_true",
                    help="skip the shape x sparsity sweep (matrix-size table A-F x 0-87.5 %%)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-roofs", action="store_true", help="skip the roof micro-benchmarks")
    ap.add_argument("--launches-only", type=int, default=0, metavar="L",
                    help="run L untimed launches of the workload and exit (for counter passes)")
    ap.add_argument("--copy-only", type=int, default=0, metavar="L",
                    help="run L plain 1 GiB device copies and exit (calibrates the HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU: the N:M SpMM path runs on a single MI355X "
              f"and has no multi-GPU mode (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py is single-process; WORLD_SIZE > 1 is not supported.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2503_01253_amd as nm
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    run = RUNS.get(args.workload) or table_runs()[args.workload]
    if args.copy_only:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(args.copy_only):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] {args.copy_only} copies of {src.numel() * 4} bytes done")
        return
    if args.launches_only:
        w = Workload(run, torch, nm)
        handle = torch.cuda.current_stream().cuda_stream
        for i in range(args.launches_only):
            w.launch(i, handle)
        torch.cuda.synchronize()
        log(f"[bench] {args.launches_only} launches of {run.name} ({w.kernel_label()}) done")
        return
    log(f"[bench] headline {run.describe()} steps={args.steps} warmup={args.warmup}")
    head, w = measure(torch, nm, run, args.steps, args.warmup, with_dense=True, graph=run.m <= 256)
    log(f"[bench] {json.dumps(head)}")

    achieved = run.useful_flops / (head["kernel_ms_mean"] * 1e-3) / 1e12
    sha = kernel_source_sha(head["kernel"])
    tr = TRAFFIC.get((run.name, head["kernel"], sha))
    tr = traffic_bytes(tr) if tr else None
    roofline = {
        "bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
        "frac": achieved / PEAK_FP32_TFLOPS, "traffic": tr,
        "traffic_unit": "bytes per launch, rocprofv3 FETCH_SIZE + WRITE_SIZE scaled by a 1 GiB copy",
        "kernel": head["kernel"], "kernel_ms_mean": head["kernel_ms_mean"],
        "kernel_ms_p10": head["kernel_ms_p10"], "kernel_ms_p90": head["kernel_ms_p90"],
        "flops_per_launch": run.useful_flops, "alg_bytes_per_launch": run.alg_bytes,
        "kernel_src_sha": sha,
    }

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        cpu = cpu_baseline(run, w.host_A, w.host_Bp, args.cpu_seconds)
        log(f"[bench] cpu {json.dumps(cpu)}")
        one = cpu_baseline(run, w.host_A, w.host_Bp, args.cpu_seconds, threads=1)
        log(f"[bench] cpu 1 thread {json.dumps(one)}")
        cpu["one_thread"] = {"value": one["value"], "cores": 1, "sample": one["sample"]}

    roofs = None
    if not args.no_roofs:
        log("[bench] measured roofs (bench/micro)")
        roofs = measured_roofs(torch)
        log(f"[bench] roofs {json.dumps(roofs)}")

    sweep = []
    if not args.no_sweep:
        for name in ("R1", "R3a", "R3b", "R3c", "R3d", "R4", "R5a", "R5b", "R5c"):
            if name == run.name:
                continue
            r = RUNS[name]
            small = r.m <= 256
            res, _ = measure(torch, nm, r, 200 if small else 30, 5, with_dense=True, graph=small)
            log(f"[bench] sweep {json.dumps(res)}")
            sweep.append({k: (round(v, 5) if isinstance(v, float) else v) for k, v in res.items()})
            torch.cuda.empty_cache()

    table = []
    if not args.no_table:
        dense_ms = {}
        for name, r in table_runs().items():
            shape = name.split("-")[0]
            with_dense = shape not in dense_ms
            res, _ = measure(torch, nm, r, 50, 5, with_dense=with_dense, graph=True)
            if with_dense:
                dense_ms[shape] = res["dense_matmul_ms"]
            d = dense_ms[shape]
            row = {
                "point": name, "m": r.m, "n": r.n, "k": r.k, "N": r.N, "M": r.M, "V": r.V,
                "sparsity_pct": round(100.0 * (1 - r.N / r.M), 1), "kernel": res["kernel"],
                "us": round(res["kernel_ms_median"] * 1e3, 2),
                "us_p10": round(res["kernel_ms_p10"] * 1e3, 2),
                "us_p90": round(res["kernel_ms_p90"] * 1e3, 2),
                "eff_tflops": round(res["eff_tflops"], 2),
                "frac_fp32_peak": round(res["eff_tflops"] / PEAK_FP32_TFLOPS, 4),
                "dense_fp32_us": round(d * 1e3, 2),
                "speedup_vs_dense": round(d / res["kernel_ms_median"], 3),
                "ideal_speedup": r.M / r.N,
            }
            log(f"[bench] table {json.dumps(row)}")
            table.append(row)
            torch.cuda.empty_cache()

    extras = {}
    if not args.no_sweep:
        log("[bench] epilogue, device packer and Eq. 2 confusion matrix")
        extras = measure_extras(torch, nm)
        log(f"[bench] extras {json.dumps(extras)}")

    ms = head["ms_per_step"]
    line = {
        "metric": "effective TFLOPS (2*m*n*k*N/M)",
        "value": run.useful_flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOPS",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {
            "workload": (f"m=n=k=4096 fp32, A,B ~ U[-1,1], vector-wise {run.N}:{run.M} "
                         f"({100 * (1 - run.N / run.M):.1f}% sparse), V={run.V}")
            if run.name == "R2" else run.describe(),
            "m": run.m, "n": run.n, "k": run.k, "N": run.N, "M": run.M, "V": run.V,
            "seed": run.seed, "parallelism": "single GPU", "cold_cache_copies": head["copies"],
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "dense_fp32_matmul": {"ms": head["dense_matmul_ms"], "speedup": head["speedup_vs_dense"],
                              "ideal_speedup": head["ideal_speedup"]},
        "paper_context": {"hardware": "NVIDIA A100 80GB PCIe (clock locked, 14.7 TFLOPS fp32 peak)",
                          "workload": "m=n=k=4096, vector length not stated",
                          "pct_of_fp32_peak_50_62.5_75_87.5": [96, 93, 95, 88]},
        "shape_sparsity_table": table,
        "sweep": sweep,
        **extras,
        "device": torch.cuda.get_device_name(0),
        "device_clocks": device_clocks(),
        "measured_roofs": roofs,
        # last, so that a reader of the line's tail sees every workload
        "summary_cols": ["run", "kernel", "us", "eff_tflops", "roof_frac", "bound", "roof_frac_measured",
                         "x_dense_fp32", "ideal_M_over_N"],
        "summary": [summary_row(r, roofs) for r in [head] + sweep],
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
