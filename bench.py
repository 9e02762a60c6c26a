"""Throughput of the segment-reduction hot path on one MI355X.

One step = one geot_segment_reduce (sum) over the power-law graph workload
(src [114,615,892 x 32] fp32, 232,965 segments with lognormal(5.5, 1.2)
lengths) plus one geot_gather_scatter (sum) over the SpMM workload (X
[2,449,029 x 128] fp32, 61,859,140 edges with Zipf(2.0) row lengths, uniform
columns, U(0,1) weights). Inputs are synthetic (seeded generators in
``workloads``) and resident in HBM before timing starts.

The metric is effective HBM bandwidth: algorithmic bytes per step divided by
the time per step, where algorithmic bytes are
  segment_reduce: nnz*F*4 (src) + nnz*8 (index) + S*F*4 (out)
  gather_scatter: nnz*(8 col + 4 weight + 8 row) + nnz*F*4 (gathered X rows) + R*F*4 (out)

Prints ONE JSON line. ``roofline`` describes the dominant kernel (the main
kernel of the call that takes longest), timed per launch with HIP events on
the stream it runs on; ``traffic`` comes from committed rocprofv3 counter
readings (profiles/traffic.json) and is null when the kernel source changed
since. ``cpu_baseline`` times the CPU oracle on a bounded sample of the same
inputs on the host (one thread), and the multi-threaded oracle over both whole
workloads on the host's cores, with the core count and CPU model.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "segment_reduce / gather_scatter effective HBM GB/s and % of MI355X HBM peak"
KERNEL_SOURCES = ("paper_2404_03019_amd/csrc/ep_kernel.h", "paper_2404_03019_amd/csrc/ep_f32_i64.hip",
                  "paper_2404_03019_amd/csrc/common.h", "paper_2404_03019_amd/csrc/internal.h")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def seg_bytes(nnz, S, F, esize=4, isize=8):
    """src + index + out; esize / isize: bytes per stored element / per id"""
    return nnz * F * esize + nnz * isize + S * F * 4


def gather_bytes(nnz, R, F, esize=4, isize=8):
    """col + weight + row per edge, one gathered X row per edge, out"""
    return nnz * (isize + 4 + isize) + nnz * F * esize + R * F * 4


def load_traffic(kernel_key: str):
    """Counter-derived HBM bytes per launch for kernel_key, if taken on the current source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    e = d.get(kernel_key)
    if not e or e.get("source_hash") != kernel_source_hash():
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(c3, c4, target_s: float):
    """The oracle (serial C, fp64 accumulation) on the first segments of each workload.

    A 1% sample is timed first; the sample is then grown so the timed oracle
    work lasts about ``target_s`` seconds (capped at the whole workload)."""
    import numpy as np

    import oracle

    oracle.default()

    def run(frac):
        L3, L4 = c3["lengths"], c4["lengths"]
        s3 = max(1, int(L3.size * frac))
        s4 = max(1, int(L4.size * frac))
        n3, n4 = int(L3[:s3].sum()), int(L4[:s4].sum())
        src = c3["src"][:n3]
        idx3 = c3["index"][:n3]
        col, w, row = c4["col"][:n4], c4["weight"][:n4], c4["index"][:n4]
        t0 = time.perf_counter()
        oracle.segment_reduce(src, idx3, s3, "sum")
        t1 = time.perf_counter()
        oracle.gather_scatter(c4["X"], col, w, row, s4, "sum")
        t2 = time.perf_counter()
        return dict(s3=s3, n3=n3, s4=s4, n4=n4, t3=t1 - t0, t4=t2 - t1,
                    bytes=seg_bytes(n3, s3, 32) + gather_bytes(n4, s4, 128))

    probe = run(0.01)
    frac = min(1.0, 0.01 * target_s / max(probe["t3"] + probe["t4"], 1e-3))
    r = run(frac) if frac > 0.01 else probe
    # the same definitions with the output segments split across host threads
    # (oracle/geot_oracle_mt.c, bit-identical results), over both whole workloads
    m = oracle.mt()
    t0 = time.perf_counter()
    m.segment_reduce(c3["src"], c3["index"], c3["num_segments"], "sum")
    t1 = time.perf_counter()
    m.gather_scatter(c4["X"], c4["col"], c4["weight"], c4["index"], c4["num_segments"], "sum")
    t2 = time.perf_counter()
    b_all = seg_bytes(c3["index"].size, c3["num_segments"], 32) + \
        gather_bytes(c4["index"].size, c4["num_segments"], 128)
    return {
        "value": round(r["bytes"] / (r["t3"] + r["t4"]) / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"first {r['s3']} of 232,965 segments of the power-law graph ({r['n3']} rows, "
                   f"{r['t3']:.1f} s) + first {r['s4']} of 2,449,029 rows of the SpMM workload "
                   f"({r['n4']} edges, {r['t4']:.1f} s); serial C oracle on one host thread; "
                   f"same algorithmic-byte formulas as the GPU value"),
        "all_cores": {
            "value": round(b_all / (t2 - t0) / 1e9, 3),
            "unit": "GB/s",
            "cores": m.threads,
            "sample": (f"both whole workloads ({t1 - t0:.1f} s + {t2 - t1:.1f} s): the oracle's definitions "
                       f"with output segments split across {m.threads} POSIX threads"),
        },
        "nproc": os.cpu_count(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": cpu_model(),
    }


def cpu_configs():
    """The oracle on every named workload on the host: one line per workload with the serial
    oracle's time (one host thread) and the threaded oracle's (one thread per CPU this process
    may run on), both with the GPU value's algorithmic-byte formulas. The CPU baseline per
    workload; it loads no GPU code."""
    import numpy as np

    import oracle
    from workloads import make_config
    from workloads.generators import C2_FEATURES

    ser, mt = oracle.default(), oracle.mt()
    host = {"nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model()}

    def secs(fn, reps):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts))

    def line(name, nbytes, fn_ser, fn_mt):
        reps = 1 if nbytes >= 1e9 else 3   # median of 3 below 1 GB
        ts, tm = secs(fn_ser, reps), secs(fn_mt, reps)
        rec = {"cpu": name, "algorithmic_bytes": nbytes, "repetitions": reps,
               "serial_s": round(ts, 5), "serial_GB/s": round(nbytes / ts / 1e9, 3),
               "threads": mt.threads, "threaded_s": round(tm, 5), "threaded_GB/s": round(nbytes / tm / 1e9, 3)}
        rec.update(host)
        print(json.dumps(rec), flush=True)

    def seg(name, src, idx, S, op):
        F = src.shape[1]
        line(name, seg_bytes(idx.size, S, F), lambda: ser.segment_reduce(src, idx, S, op),
             lambda: mt.segment_reduce(src, idx, S, op))

    c = make_config("c1_zipf_small")
    seg("c1_zipf_small sum", c["src"], c["index"], c["num_segments"], "sum")
    c = make_config("c2_poisson_fsweep", F=256)
    for F in C2_FEATURES:
        src = np.ascontiguousarray(c["src"][:, :F])
        for op in ("sum", "mean", "max"):
            seg(f"c2_poisson_fsweep F={F} {op}", src, c["index"], c["num_segments"], op)
    del c, src
    c = make_config("c5_pointcloud_knn")
    for op in ("mean", "max"):
        seg(f"c5_pointcloud_knn {op}", c["src"], c["index"], c["num_segments"], op)
    del c
    c = make_config("c3_powerlaw_graph")
    seg("c3_powerlaw_graph sum", c["src"], c["index"], c["num_segments"], "sum")
    del c
    c = make_config("c4_spmm")
    R = c["num_segments"]
    line("c4_spmm sum", gather_bytes(c["index"].size, R, 128),
         lambda: ser.gather_scatter(c["X"], c["col"], c["weight"], c["index"], R, "sum"),
         lambda: mt.gather_scatter(c["X"], c["col"], c["weight"], c["index"], R, "sum"))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_probe(n: int):
    """A plain copy of known size: 2 GiB read and 2 GiB written per launch."""
    import torch

    a = torch.ones(1 << 29, device="cuda:0")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        b.copy_(a)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / n
    print(json.dumps({"copy_bytes_read": 1 << 31, "copy_bytes_written": 1 << 31,
                      "ms_per_copy": round(dt * 1e3, 4),
                      "GB/s": round(2 * (1 << 31) / dt / 1e9, 1)}), flush=True)


def profile_configs(reps: int):
    """Each named workload's main calls, `reps` times each, for counter and kernel-trace runs
    (rocprofv3 --pmc FETCH_SIZE, --pmc WRITE_SIZE, --kernel-trace). Before the calls of the
    k-th entry a marker runs: a segment reduction with no rows over 2048 * (k + 1) segments of
    one column, i.e. one fill kernel of k + 1 blocks, and after them one of 1,000 blocks, so
    the dispatches between the two belong to entry k. The entries, in order, are printed as
    JSON lines."""
    import numpy as np
    import torch

    import paper_2404_03019_amd as geot
    from workloads import make_config

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    geot.lib()
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    e_src = torch.empty((0, 1), device=dev)
    e_idx = torch.empty(0, dtype=torch.int64, device=dev)
    entries = []

    def entry(name, nbytes, fn):
        k = len(entries)
        torch.cuda.synchronize()
        geot.segment_reduce(e_src, e_idx, 2048 * (k + 1), "sum")
        for _ in range(reps):
            fn()
        geot.segment_reduce(e_src, e_idx, 2048 * 1000, "sum")   # end marker: 1,000 blocks
        torch.cuda.synchronize()
        entries.append(name)
        print(json.dumps({"entry": k, "name": name, "algorithmic_bytes": nbytes, "calls": reps,
                          "choice": geot.last_choice()}), flush=True)

    a = torch.ones(1 << 29, device=dev)
    b = torch.empty_like(a)
    entry("plain copy of 2 GiB (calibration)", 2 * (1 << 31), lambda: b.copy_(a))
    del a, b
    c = make_config("c1_zipf_small")
    s, i = up(c["src"]), up(c["index"])
    entry("c1_zipf_small sum", seg_bytes(i.numel(), 4096, 32), lambda: geot.segment_reduce(s, i, 4096, "sum"))
    c = make_config("c2_poisson_fsweep", F=256)
    i = up(c["index"])
    for F in (1, 3, 4, 15, 16, 64, 256):
        s = up(c["src"][:, :F])
        entry(f"c2_poisson_fsweep F={F} sum", seg_bytes(i.numel(), 100_000, F),
              lambda: geot.segment_reduce(s, i, 100_000, "sum"))
    del c, s, i
    c = make_config("c5_pointcloud_knn")
    s, i = up(c["src"]), up(c["index"])
    for op in ("mean", "max"):
        entry(f"c5_pointcloud_knn {op}", seg_bytes(i.numel(), 1_048_576, 64),
              lambda: geot.segment_reduce(s, i, 1_048_576, op))
    del c, s, i
    torch.cuda.empty_cache()
    c3 = make_config("c3_powerlaw_graph")
    S3 = c3["num_segments"]
    s, i = up(c3["src"]), up(c3["index"])
    n3 = i.numel()
    del c3
    entry("c3_powerlaw_graph sum", seg_bytes(n3, S3, 32), lambda: geot.segment_reduce(s, i, S3, "sum"))
    s16, i32 = s.to(torch.bfloat16), i.to(torch.int32)
    entry("c3_powerlaw_graph sum bf16 int32", seg_bytes(n3, S3, 32, 2, 4),
          lambda: geot.segment_reduce(s16, i32, S3, "sum"))
    del s16, i32
    g3 = torch.randn(S3, 32, device=dev)
    gs = torch.empty_like(s)
    for op in ("sum", "mean", "max"):
        o = geot.segment_reduce(s, i, S3, op)
        nb = n3 * 8 + n3 * 128 + S3 * 128 + (n3 * 128 + S3 * 128 if op == "max" else 0)
        entry(f"c3_powerlaw_graph gradient {op}", nb,
              lambda: geot.segment_reduce_backward(g3, i, op, s, o, grad_src=gs))
    entry("c3_powerlaw_graph max with recipients", seg_bytes(n3, S3, 32) + S3 * 128,
          lambda: geot.segment_reduce_max_arg(s, i, S3))
    _, a3 = geot.segment_reduce_max_arg(s, i, S3)
    entry("c3_powerlaw_graph gradient max from recorded recipients", n3 * 8 + n3 * 128 + 2 * S3 * 128,
          lambda: geot.segment_reduce_backward_max_arg(g3, i, a3))
    del s, i, g3, gs, o, a3
    torch.cuda.empty_cache()
    c4 = make_config("c4_spmm")
    R4 = c4["num_segments"]
    X, col, w, row = up(c4["X"]), up(c4["col"]), up(c4["weight"]), up(c4["index"])
    n4 = row.numel()
    del c4
    entry("c4_spmm sum", gather_bytes(n4, R4, 128), lambda: geot.gather_scatter(X, col, w, row, R4, "sum"))
    X16, c32, r32 = X.to(torch.bfloat16), col.to(torch.int32), row.to(torch.int32)
    entry("c4_spmm sum bf16 int32", gather_bytes(n4, R4, 128, 2, 4),
          lambda: geot.gather_scatter(X16, c32, w, r32, R4, "sum"))
    del X16, c32, r32
    g4 = torch.randn(R4, 128, device=dev)
    entry("c4_spmm gradient grad_X sum", n4 * 20 + n4 * 512 + R4 * 512,
          lambda: geot.gather_scatter_backward(X, col, w, row, g4, "sum", need_weight=False))
    entry("c4_spmm gradient grad_weight sum", n4 * 20 + n4 * 512 + R4 * 512,
          lambda: geot.gather_scatter_backward(X, col, w, row, g4, "sum", need_x=False))
    entry("c4_spmm transpose_edges", n4 * 40, lambda: geot.transpose_edges(col, w, row, R4, R4, "sum"))
    o4 = geot.gather_scatter(X, col, w, row, R4, "max")
    entry("c4_spmm gradient max", 3 * (n4 * 20 + n4 * 512 + R4 * 512),
          lambda: geot.gather_scatter_backward(X, col, w, row, g4, "max", out=o4))
    entry("c4_spmm max with recipients", gather_bytes(n4, R4, 128) + R4 * 512,
          lambda: geot.gather_scatter_max_arg(X, col, w, row, R4))
    _, a4 = geot.gather_scatter_max_arg(X, col, w, row, R4)
    entry("c4_spmm gradient max from recorded recipients", 2 * (n4 * 20 + n4 * 512 + R4 * 512),
          lambda: geot.gather_scatter_backward_max_arg(X, col, w, row, g4, a4))


# the per-edge byte count of a gather over the transposed list charges every gathered row; those
# are the destination rows of a power-law graph, which repeat and mostly hit in cache, so the
# rate can exceed the HBM peak and is no HBM rate there
GATHER_REUSE = "gathered rows repeat (cache hits): the per-edge rate exceeds HBM; see compulsory_bytes"


def suite(reps: int):
    """One JSON line per measurement: every named workload and op, the gradients on the two
    large workloads, and a two-layer graph-convolution training step (library autograd vs the
    same model with torch's index_add). Median over `reps` HIP-event timings per entry; for
    inputs under 1 GB a 512 MB read evicts them from the MALL before each repetition (a read,
    so no dirty lines are written back inside the timed call)."""
    import numpy as np
    import torch

    import paper_2404_03019_amd as geot
    import paper_2404_03019_amd.autograd as ga
    from workloads import make_config
    from workloads.generators import C2_FEATURES

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    geot.lib()
    flush = torch.ones(1 << 27, device=dev)

    def timed(fn, nbytes_in):
        cold = nbytes_in < (1 << 30)
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            if cold:
                flush.sum()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts)), cold

    def emit(name, ms, nbytes, cold, **extra):
        rec = {"suite": name, "ms": round(ms, 4), "algorithmic_bytes": nbytes,
               "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
               "pct_of_hbm_peak": round(100 * nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 1),
               "mall_flushed": cold, "choice": geot.last_choice()}
        rec.update(extra)
        print(json.dumps(rec), flush=True)

    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    # segment reductions
    c = make_config("c1_zipf_small")
    src, idx = up(c["src"]), up(c["index"])
    b = seg_bytes(idx.numel(), c["num_segments"], 32)
    ms, cold = timed(lambda: geot.segment_reduce(src, idx, c["num_segments"], "sum"), b)
    emit("c1_zipf_small sum", ms, b, cold)
    c = make_config("c2_poisson_fsweep", F=256)
    idx = up(c["index"])
    st2 = geot.index_stats(idx, c["num_segments"])
    for F in C2_FEATURES:
        src = up(c["src"][:, :F])
        b = seg_bytes(idx.numel(), c["num_segments"], F)
        for op in ("sum", "mean", "max"):
            ms, cold = timed(lambda: geot.segment_reduce(src, idx, c["num_segments"], op), b)
            emit(f"c2_poisson_fsweep F={F} {op}", ms, b, cold)
        # with the index's length statistics (kept by the caller): the selector sees the spread
        ms, cold = timed(lambda: geot.segment_reduce(src, idx, c["num_segments"], "sum", stats=st2), b)
        emit(f"c2_poisson_fsweep F={F} sum, with index statistics", ms, b, cold)
        del src
    del c
    c = make_config("c5_pointcloud_knn")
    src, idx = up(c["src"]), up(c["index"])
    b = seg_bytes(idx.numel(), c["num_segments"], 64)
    st5 = geot.index_stats(idx, c["num_segments"])
    for op in ("mean", "max"):
        ms, cold = timed(lambda: geot.segment_reduce(src, idx, c["num_segments"], op), b)
        emit(f"c5_pointcloud_knn {op}", ms, b, cold)
        ms, cold = timed(lambda: geot.segment_reduce(src, idx, c["num_segments"], op, stats=st5), b)
        emit(f"c5_pointcloud_knn {op}, with index statistics", ms, b, cold)
    del src, idx, c
    torch.cuda.empty_cache()
    # the two large workloads, forward and gradients
    c3 = make_config("c3_powerlaw_graph")
    S3 = c3["num_segments"]
    src, idx = up(c3["src"]), up(c3["index"])
    n3 = idx.numel()
    b = seg_bytes(n3, S3, 32)
    ms, cold = timed(lambda: geot.segment_reduce(src, idx, S3, "sum"), b)
    emit("c3_powerlaw_graph sum", ms, b, cold)
    ms, _ = timed(lambda: geot.index_stats(idx, S3), 1 << 40)
    emit("c3_powerlaw_graph index statistics (geot_index_stats, synchronizing)", ms, n3 * 8 + (S3 + 1) * 8, False)
    # the same reduction with bf16 storage and int32 ids (fp32 accumulation and output)
    src16, idx32 = src.to(torch.bfloat16), idx.to(torch.int32)
    b = seg_bytes(n3, S3, 32, 2, 4)
    ms, cold = timed(lambda: geot.segment_reduce(src16, idx32, S3, "sum"), b)
    emit("c3_powerlaw_graph sum bf16 int32", ms, b, cold)
    del src16, idx32
    g3 = torch.randn(S3, 32, device=dev)
    gsrc = torch.empty_like(src)
    for op in ("sum", "mean", "max"):
        out = geot.segment_reduce(src, idx, S3, op)
        # bytes: index + grad_src written + grad_out read; max also reads src and out per row
        b = n3 * 8 + n3 * 128 + S3 * 128 + (n3 * 128 + S3 * 128 if op == "max" else 0)
        ms, cold = timed(lambda: geot.segment_reduce_backward(g3, idx, op, src, out, grad_src=gsrc), b)
        emit(f"c3_powerlaw_graph backward {op}", ms, b, cold)
    del gsrc
    # max recording its recipients (the forward writes a uint32 per output element besides
    # out), then the gradient from them: one pass that writes grad_src (index + grad_src
    # written + grad_out and the recipients read)
    b = seg_bytes(n3, S3, 32) + S3 * 128
    ms, cold = timed(lambda: geot.segment_reduce_max_arg(src, idx, S3), b)
    emit("c3_powerlaw_graph max with recipients", ms, b, cold)
    _, arg3 = geot.segment_reduce_max_arg(src, idx, S3)
    b = n3 * 8 + n3 * 128 + 2 * S3 * 128
    ms, cold = timed(lambda: geot.segment_reduce_backward_max_arg(g3, idx, arg3), b)
    emit("c3_powerlaw_graph backward max from recorded recipients", ms, b, cold)
    del arg3
    # the gradients with bf16 storage and int32 ids: grad_src written as bf16
    src16, idx32 = src.to(torch.bfloat16), idx.to(torch.int32)
    gsrc16 = torch.empty_like(src16)
    for op in ("sum", "mean", "max"):
        out = geot.segment_reduce(src16, idx32, S3, op)
        b = n3 * 4 + n3 * 64 + S3 * 128 + (n3 * 64 + S3 * 128 if op == "max" else 0)
        ms, cold = timed(lambda: geot.segment_reduce_backward(g3, idx32, op, src16, out, grad_src=gsrc16), b)
        emit(f"c3_powerlaw_graph backward {op} bf16 int32", ms, b, cold)
    del src16, idx32, gsrc16
    del src, idx, g3, c3
    torch.cuda.empty_cache()
    c4 = make_config("c4_spmm")
    R4 = c4["num_segments"]
    X, col, w, row = up(c4["X"]), up(c4["col"]), up(c4["weight"]), up(c4["index"])
    n4 = row.numel()
    b = gather_bytes(n4, R4, 128)
    ms, cold = timed(lambda: geot.gather_scatter(X, col, w, row, R4, "sum"), b)
    # compulsory: the edge metadata, X read once, out written
    emit("c4_spmm sum", ms, b, cold, compulsory_bytes=n4 * 20 + 2 * R4 * 512)
    X16, col32, row32 = X.to(torch.bfloat16), col.to(torch.int32), row.to(torch.int32)
    b = gather_bytes(n4, R4, 128, 2, 4)
    ms, cold = timed(lambda: geot.gather_scatter(X16, col32, w, row32, R4, "sum"), b)
    emit("c4_spmm sum bf16 int32", ms, b, cold)
    # unfused: materialise the weighted messages with torch, then reduce them (the paper's
    # motivation for fusing: the message tensor is written and read back once)
    b = gather_bytes(n4, R4, 128)

    def unfused():
        msg = torch.index_select(X, 0, col).mul_(w[:, None])
        geot.segment_reduce(msg, row, R4, "sum")
    ms_u, _ = timed(unfused, b)
    emit("c4_spmm sum unfused (torch gather + segment_reduce)", ms_u, b, False)
    g4 = torch.randn(R4, 128, device=dev)
    # the gradients with X stored as bf16 and int32 ids (fp32 gradients): the grad_X bytes
    # count 12 bytes of metadata per edge, grad_w the gathered X row at 2 bytes an element
    b = n4 * 12 + n4 * 512 + R4 * 512
    ms, cold = timed(lambda: geot.gather_scatter_backward(X16, col32, w, row32, g4, "sum", need_weight=False), b)
    emit("c4_spmm backward grad_X bf16 int32", ms, b, cold, compulsory_bytes=n4 * 12 + 2 * R4 * 512,
         note=GATHER_REUSE)
    b = n4 * 12 + n4 * 256 + R4 * 512
    ms, cold = timed(lambda: geot.gather_scatter_backward(X16, col32, w, row32, g4, "sum", need_x=False), b)
    emit("c4_spmm backward grad_weight bf16 int32", ms, b, cold)
    del X16, col32, row32
    # grad_X: edge metadata + one gathered grad_out row per edge + grad_X written; the
    # compulsory bytes read the metadata and each grad_out row once and write grad_X
    b = n4 * 20 + n4 * 512 + R4 * 512
    ms, cold = timed(lambda: geot.gather_scatter_backward(X, col, w, row, g4, "sum", need_weight=False), b)
    emit("c4_spmm backward grad_X", ms, b, cold, compulsory_bytes=n4 * 20 + 2 * R4 * 512, note=GATHER_REUSE)
    # grad_w: col, row (the weight is not read for sum) + one gathered X row per edge + each
    # grad_out row once (edges are sorted by row) + grad_w written; same count as the forward
    b = n4 * 20 + n4 * 512 + R4 * 512
    ms, cold = timed(lambda: geot.gather_scatter_backward(X, col, w, row, g4, "sum", need_x=False), b)
    emit("c4_spmm backward grad_weight", ms, b, cold)
    # max: recipients (one gathered X row per edge + out), then grad_X (the recipients' grad_out
    # rows, one atomic add each) and grad_w (one gathered X row per edge, masked): bytes of the
    # three passes' streams, atomics not counted
    out4 = geot.gather_scatter(X, col, w, row, R4, "max")
    b = 3 * (n4 * 20 + n4 * 512 + R4 * 512)
    ms, cold = timed(lambda: geot.gather_scatter_backward(X, col, w, row, g4, "max", out=out4), b)
    emit("c4_spmm backward max (grad_X and grad_weight)", ms, b, cold)
    del out4
    # max recording its recipients, then both gradients from them (no recipient pass): bytes of
    # the forward plus the recipients written; of the gradients, the weight pass's and the
    # pull's streams as above (two passes)
    b = gather_bytes(n4, R4, 128) + R4 * 512
    ms, cold = timed(lambda: geot.gather_scatter_max_arg(X, col, w, row, R4), b)
    emit("c4_spmm max with recipients", ms, b, cold)
    _, arg4 = geot.gather_scatter_max_arg(X, col, w, row, R4)
    b = 2 * (n4 * 20 + n4 * 512 + R4 * 512)
    ms, cold = timed(lambda: geot.gather_scatter_backward_max_arg(X, col, w, row, g4, arg4), b)
    emit("c4_spmm backward max from recorded recipients (grad_X and grad_weight)", ms, b, cold)
    del arg4
    # a static graph keeps its column-sorted edge list: the gradient w.r.t. X is then one gather
    ms, _ = timed(lambda: geot.transpose_edges(col, w, row, R4, R4, "sum"), 1 << 40)
    emit("c4_spmm transpose_edges (once per static graph)", ms, n4 * 40, False)
    sc, rt, cf = geot.transpose_edges(col, w, row, R4, R4, "sum")
    b = n4 * 20 + n4 * 512 + R4 * 512
    ms, _ = timed(lambda: geot.gather_scatter(g4, rt, cf, sc, R4, "sum"), 1 << 40)
    # the per-edge count charges every gathered row; these are the destination rows of a
    # power-law graph, which repeat and mostly hit in cache, so its rate is no HBM rate. The
    # compulsory bytes read each grad_out row once
    emit("c4_spmm backward grad_X from a kept transposed list", ms, b, False,
         compulsory_bytes=n4 * 20 + 2 * R4 * 512, note=GATHER_REUSE)
    del g4, sc, rt, cf
    # two-layer graph convolution training step on the SpMM graph (128 -> 128 -> 64)
    torch.manual_seed(0)
    layers = torch.nn.ModuleList([ga.GraphConv(128, 128), ga.GraphConv(128, 64)]).to(dev)
    target = torch.randn(R4, 64, device=dev)

    def step_geot():
        layers.zero_grad(set_to_none=True)
        h = torch.relu(layers[0](X, col, row, R4, w))
        loss = ((layers[1](h, col, row, R4, w) - target) ** 2).mean()
        loss.backward()

    def agg_torch(z):
        return torch.zeros(R4, z.shape[1], device=dev).index_add_(0, row, z[col] * w[:, None])

    def step_torch():
        layers.zero_grad(set_to_none=True)
        h = torch.relu(agg_torch(layers[0].lin(X)) + layers[0].bias)
        loss = ((agg_torch(layers[1].lin(h)) + layers[1].bias - target) ** 2).mean()
        loss.backward()

    # index statistics pass (the optional selector features): one read of the index
    for name, ix, S_ in (("c4_spmm", row, R4),):
        ms, _ = timed(lambda: geot.index_stats(ix, S_), 1 << 40)
        emit(f"{name} index statistics (geot_index_stats, synchronizing)", ms, ix.numel() * 8 + (S_ + 1) * 8,
             False)
    graph = ga.Graph(col, row, R4, w)

    def step_geot_graph():
        layers.zero_grad(set_to_none=True)
        h = torch.relu(layers[0](X, graph))
        loss = ((layers[1](h, graph) - target) ** 2).mean()
        loss.backward()

    ms_g, _ = timed(step_geot, 1 << 40)
    ms_c, _ = timed(step_geot_graph, 1 << 40)
    ms_t, _ = timed(step_torch, 1 << 40)
    print(json.dumps({"suite": "graphconv 2-layer training step (SpMM graph, 128-128-64)",
                      "ms": round(ms_g, 3), "torch_index_add_ms": round(ms_t, 3),
                      "speedup_vs_torch": round(ms_t / ms_g, 2)}), flush=True)
    print(json.dumps({"suite": "graphconv 2-layer training step, Graph with a kept transposed list",
                      "ms": round(ms_c, 3), "torch_index_add_ms": round(ms_t, 3),
                      "speedup_vs_torch": round(ms_t / ms_c, 2)}), flush=True)
    del layers
    # two GIN layers (learned eps) on the same graph without weights, with a kept transposed list
    gin = torch.nn.ModuleList([ga.GINConv(128, 128, train_eps=True), ga.GINConv(128, 64, train_eps=True)]).to(dev)
    graph_u = ga.Graph(col, row, R4)

    def step_gin():
        gin.zero_grad(set_to_none=True)
        h = torch.relu(gin[0](X, graph_u))
        loss = ((gin[1](h, graph_u) - target) ** 2).mean()
        loss.backward()

    def gin_torch(layer, z):
        u = (1.0 + layer.eps) * z + torch.zeros_like(z).index_add_(0, row, z[col])
        return layer.lin2(torch.relu(layer.lin1(u)))

    def step_gin_torch():
        gin.zero_grad(set_to_none=True)
        h = torch.relu(gin_torch(gin[0], X))
        loss = ((gin_torch(gin[1], h) - target) ** 2).mean()
        loss.backward()

    ms_gi, _ = timed(step_gin, 1 << 40)
    ms_gt, _ = timed(step_gin_torch, 1 << 40)
    print(json.dumps({"suite": "gin 2-layer training step (SpMM graph without weights, 128-128-64, kept list)",
                      "ms": round(ms_gi, 3), "torch_index_add_ms": round(ms_gt, 3),
                      "speedup_vs_torch": round(ms_gt / ms_gi, 2)}), flush=True)
    host_probe()


def host_probe():
    """Selector host cost per call and the HBM peak from device properties (a small host
    program linked against the library, built here with hipcc)."""
    import subprocess
    exe = os.path.join(ROOT, "_build", "host_probe")
    os.makedirs(os.path.dirname(exe), exist_ok=True)
    lib_dir = os.path.join(ROOT, "paper_2404_03019_amd")
    subprocess.run(["/opt/rocm/bin/hipcc", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
                    os.path.join(lib_dir, "tune", "host_probe.cpp"), f"-L{lib_dir}", "-lgeot_hip",
                    f"-Wl,-rpath,{lib_dir}", "-o", exe], check=True, capture_output=True)
    r = subprocess.run([exe], check=True, capture_output=True, text=True)
    print(r.stdout.strip(), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate host seconds of oracle work for cpu_baseline")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="N",
                    help="only run N plain device copies of 2 GiB (calibrates HBM byte counters)")
    ap.add_argument("--profile-configs", type=int, default=0, metavar="N",
                    help="only run every named workload's main calls N times each, behind markers, "
                         "for rocprofv3 counter and kernel-trace runs")
    ap.add_argument("--suite", action="store_true",
                    help="instead of the headline line: one line per workload, op and gradient")
    ap.add_argument("--cpu-configs", action="store_true",
                    help="only the CPU baseline per named workload: the serial and the threaded oracle")
    args = ap.parse_args()
    if args.cpu_configs:
        cpu_configs()
        return
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.profile_configs:
        profile_configs(args.profile_configs)
        return
    if args.suite:
        suite(max(3, args.steps))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the path does not shard across GPUs); "
              f"got --gpus {args.gpus}", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1 or args.warmup < 0:
        sys.exit("steps must be >= 1 and warmup >= 0")

    import numpy as np
    import torch

    import paper_2404_03019_amd as geot
    from workloads import make_config

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    geot.lib()  # fail loudly if the library is missing

    log("generating power-law graph workload")
    c3 = make_config("c3_powerlaw_graph")
    log("generating SpMM workload")
    c4 = make_config("c4_spmm")
    S3, F3, n3 = c3["num_segments"], 32, c3["index"].size
    R4, F4, n4 = c4["num_segments"], 128, c4["index"].size
    log("uploading")
    src = torch.from_numpy(c3["src"]).to(dev)
    idx = torch.from_numpy(c3["index"]).to(dev)
    X = torch.from_numpy(c4["X"]).to(dev)
    col = torch.from_numpy(c4["col"]).to(dev)
    w = torch.from_numpy(c4["weight"]).to(dev)
    row = torch.from_numpy(c4["index"]).to(dev)
    out3 = torch.empty((S3, F3), device=dev)
    out4 = torch.empty((R4, F4), device=dev)
    torch.cuda.synchronize()

    b3 = seg_bytes(n3, S3, F3)
    b4 = gather_bytes(n4, R4, F4)

    def step():
        geot.segment_reduce(src, idx, S3, "sum", out=out3)
        geot.gather_scatter(X, col, w, row, R4, "sum", out=out4)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    choice3 = geot.select(n3, S3, F3, "sum")
    choice4 = geot.select(n4, R4, F4, "sum", gather=True)

    # timed region: exactly `steps` steps, main-kernel durations recorded by HIP events
    geot.profile_begin(2 * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    durs = geot.profile_end(2 * args.steps)
    elapsed_ms = (t1 - t0) * 1e3
    ms_per_step = elapsed_ms / args.steps
    value = (b3 + b4) / (ms_per_step * 1e-3) / 1e9

    k3 = durs[0::2]
    k4 = durs[1::2]
    avg3 = float(np.mean(k3))
    avg4 = float(np.mean(k4))
    if avg4 >= avg3:
        dom_key, dom_bytes, dom_ms, dom_name = "ep_kernel/gather/c4_spmm", b4, avg4, "gather_scatter main kernel"
    else:
        dom_key, dom_bytes, dom_ms, dom_name = "ep_kernel/rows/c3_powerlaw_graph", b3, avg3, "segment_reduce main kernel"
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    traffic = load_traffic(dom_key)

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded generators; the paper's datasets are not used)",
        "config": {
            "workload": ("power-law graph segment_reduce sum [114,615,892 x 32], 232,965 segments "
                         "+ SpMM gather_scatter sum X [2,449,029 x 128], 61,859,140 edges"),
            "bytes_per_step": b3 + b4,
            "parts": [
                {"op": "segment_reduce sum", "bytes": b3, "main_kernel_ms": round(avg3, 4),
                 "GB/s": round(b3 / (avg3 * 1e-3) / 1e9, 1), "choice": choice3},
                {"op": "gather_scatter sum", "bytes": b4, "main_kernel_ms": round(avg4, 4),
                 "GB/s": round(b4 / (avg4 * 1e-3) / 1e9, 1), "choice": choice4},
            ],
            "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 1),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": dom_name,
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": dom_bytes,
            "avg_launch_ms": round(dom_ms, 4),
        },
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        del src, idx, X, col, w, row
        torch.cuda.empty_cache()
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(c3, c4, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
