"""Throughput of the fused encode + lookup-accumulate path on one MI355X.

A step is one call of the fused path (maddness_matmul: tree encoding of
every row plus int8 lookup-accumulate and dequantization) over the whole
batch of the conv3x3_im2col workload (N = 131072 rows, D = 576, C = 32
codebooks, M = 64 outputs), inputs already resident in HBM.  Prints one JSON
line with rows/s, the HBM roofline of the fused kernel, the CPU oracle timed
on a bounded sample of the same workload, and a dense fp32 GEMM of the same
shape as context.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]

The timed outputs are checked against the CPU oracle in the same run (every
row of the headline workload), and the line's `context.workloads` block gives
the other four workloads (classifier_tiny, dense_hidden, wide_layer,
encode_heavy_f32) a compact measurement each: rows/s, step time, HBM
fraction, the accumulate's LDS fraction and a parity check on sampled rows.

Other workloads (--workload) time the same step on their shapes as the main
line; their tables are larger than LDS (the tiny classifier's aside), so a
step is an encode launch plus an accumulate launch (the row-uniform kernel
for tables at least 512 int8 or 256 fp32 columns wide, the column-tiled one
otherwise).
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
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, published
LDS_PEAK_TBS = 157.3   # 256 B/clk per CU x 256 CUs x 2.4 GHz (a ds_read_b128 probe reaches about 88% of it)
I8_MFMA_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix-core peak, published (5.0 POP/s)
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of what defines the timed kernel: its source file, its argument
    struct and the planner that picks its launch shape."""
    csrc = os.path.join(ROOT, "paper_2207_05808_amd", "csrc")

    def block(text, start, end):
        i = text.index(start)
        return text[i:text.index(end, i) + len(end)]

    h = hashlib.sha256()
    with open(os.path.join(csrc, "fused_gather.hip"), "rb") as fh:
        h.update(fh.read())
    internal = open(os.path.join(csrc, "internal.hpp")).read()
    h.update(block(internal, "struct GArgs {", "};").encode())
    api = open(os.path.join(csrc, "api.hip")).read()
    h.update(block(api, "bool plan_gfused(", "\n}\n").encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(spec, N) -> int:
    """Bytes the fused path must move per launch, each counted once: every row
    of A (4 D bytes; the split columns touch every 64-byte segment of a row),
    every output (4 M bytes), the table (16 C M entries, int8 or fp32), the
    trees (4 split ints + 15 thresholds per codebook) and, for int8 tables,
    the scales and offsets."""
    per_row = 4 * spec.D + 4 * spec.M
    entry = 1 if spec.quantized else 4
    fixed = 16 * spec.C * spec.M * entry + spec.C * (4 * 4 + 15 * 4) + (2 * 4 * spec.C if spec.quantized else 0)
    return N * per_row + fixed


def a_coverage(split, D, lda, rows=256):
    """Share of the 32-byte sectors, 64-byte segments and 128-byte lines
    spanned by a row of A that the split columns touch (over the first rows,
    each at its own offset lda * 4 bytes in): how much of every row the
    encode must fetch from HBM whatever it does."""
    cols = np.unique(np.minimum(np.asarray(split).ravel(), D - 1)).astype(np.int64)
    out = {}
    for size, key in ((32, "sector32"), (64, "segment64"), (128, "line128")):
        touched = spanned = 0
        for r in range(rows):
            base = r * lda * 4
            touched += len(np.unique((base + 4 * cols) // size))
            spanned += (base + 4 * D - 1) // size - base // size + 1
        out[key] = round(touched / spanned, 4)
    return out


def stored_traffic(workload: str, kh: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when it is missing or was taken on a different kernel source."""
    path = os.path.join(PROFILE_DIR, f"traffic_fused_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_hash") != kh:
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def _oracle_path(p):
    """The oracle's whole path for workload p: a function of rows of A."""
    import oracle
    o = oracle.get()
    if p.spec.quantized:
        lut, scale, offset = o.build_quantized_lut(p.P, p.B)
        return o, (lambda A: o.matmul(A, p.split, p.thr, lut, scale, offset)[2]), "int8"
    lut = o.build_lut_f32(p.P, p.B)
    return o, (lambda A: o.matmul_f32(A, p.split, p.thr, lut)[1]), "fp32"


def _timed_passes(run, A, rows, budget_s):
    done, passes = 0, 0
    t = time.perf_counter()
    while True:
        run(A[:rows])
        done += rows
        passes += 1
        if time.perf_counter() - t >= budget_s:
            break
    return done, passes, time.perf_counter() - t


def cpu_baseline(p, budget_s: float, one_core_s: float):
    """The oracle as it stands, timed on whole passes over the workload's rows
    (or a prefix of them, if one pass would exceed the budget) until about
    `budget_s` seconds of host time have been spent, on all the host threads
    it uses; then on one thread over the first min(N, 8192) rows for about
    `one_core_s` seconds."""
    o, run, what = _oracle_path(p)
    probe = min(p.N, 256 if p.spec.C * p.spec.M > 100000 else 2048)
    t = time.perf_counter()
    run(p.A[:probe])
    per_row = max((time.perf_counter() - t) / probe, 1e-9)
    rows = int(min(p.N, max(probe, budget_s / per_row)))
    done, passes, dt = _timed_passes(run, p.A, rows, budget_s)
    threads = o.max_threads()
    out = {"value": done / dt, "unit": "rows/s", "cores": threads, "kind": "oracle",
           "sample": f"{passes} pass(es) over the first {rows} of {p.N} rows, full encode + "
                     f"{what} lookup-accumulate, {dt:.1f} s wall"}
    rows1 = min(p.N, 8192)
    o.set_threads(1)
    try:
        d1, n1, t1 = _timed_passes(run, p.A, rows1, one_core_s)
    finally:
        o.set_threads(threads)
    out["one_core"] = {"value": d1 / t1, "unit": "rows/s", "cores": 1,
                       "sample": f"{n1} pass(es) over the first {rows1} rows, {t1:.1f} s wall"}
    return out


def parity_report(p, y_host, rows, run=None):
    """The timed outputs of `rows` against the oracle's path on the same rows:
    bit-identical outputs (the bar is 1e-6 relative) and the largest
    relative difference."""
    if run is None:
        _, run, _ = _oracle_path(p)
    ref = run(p.A[rows])
    y = y_host[rows] if y_host.shape[0] != len(rows) else y_host
    d = np.abs(y.astype(np.float64) - ref.astype(np.float64))
    rel = d / np.maximum(np.abs(ref.astype(np.float64)), np.finfo(np.float32).tiny)
    mx = float(rel.max(initial=0.0))
    return {"rows_checked": int(len(rows)), "of_rows": int(p.N), "y_bit_identical": bool(np.array_equal(y, ref)),
            "max_rel_err": mx, "ok": bool(mx <= 1e-6)}


def sampled_rows(N, n=2048, seed=0):
    """First and last n/4 rows and n/2 uniformly drawn rows."""
    rng = np.random.default_rng(seed)
    q = n // 4
    rows = set(range(min(N, q))) | set(range(max(0, N - q), N)) | set(int(r) for r in rng.integers(0, N, size=n // 2))
    return np.array(sorted(rows))


def region_us(fn, stream, reps=20, warm=3):
    """Average duration of one call of fn(i), from one event pair on the
    launch stream around `reps` back-to-back calls (after `warm` calls)."""
    import torch
    for i in range(warm):
        fn(i)
    torch.cuda.synchronize()
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    r0.record(stream)
    for i in range(reps):
        fn(i)
    r1.record(stream)
    torch.cuda.synchronize()
    return r0.elapsed_time(r1) / reps * 1e3


def repeat_us(fn, stream, reps, blocks=5):
    """Minimum and median over `blocks` repeats of the average duration of one
    call of fn(i) in `reps` back-to-back calls (one event pair per repeat: an
    event pair around every call would add its own overhead to each)."""
    import torch
    d = []
    for _ in range(blocks):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for i in range(reps):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        d.append(a.elapsed_time(b) * 1e3 / reps)
    d.sort()
    return d[0], float(np.median(d))


def copy_peak_gbs(dev, mb=512, reps=10):
    """Device-to-device copy rate of an mb-MiB buffer (bytes read + written per
    second): a measured practical peak of the HBM beside the published one."""
    import torch
    src = torch.ones((mb << 20) // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream()
    us = region_us(lambda i: dst.copy_(src), stream, reps=reps, warm=3)
    del src, dst
    return 2.0 * (mb << 20) / (us * 1e-6) / 1e9


WARM_SECONDS = 0.2   # minimum warm-up of each workload block


def onehot_product_route(spec, N):
    """Whether the library's accumulate takes the one-hot int8 product for
    this layer (int8 table, C % 16 == 0, C <= 128, M % 4 == 0, 16384 rows or
    more; the buffers here are aligned): for reporting its roof only."""
    return spec.quantized and spec.C % 16 == 0 and spec.C <= 128 and spec.M % 4 == 0 and N >= 16384


def workload_block(name, steps, warmup, sample_n=2048):
    """Compact measurement of one workload's step (the fused entry point over
    all its rows, inputs resident): rows/s, step time, HBM fraction of the
    algorithmic bytes, encode and accumulate alone, the accumulate's LDS
    fraction (two-phase shapes), a dense fp32 GEMM of the same shape, and the
    timed outputs against the oracle (every row of the tiny classifier, else
    `sample_n` rows)."""
    import torch
    import paper_2207_05808_amd as mdn
    from paper_2207_05808_amd import workloads as W
    spec = W.SPECS[name]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    log(f"[bench] workload {name}: N={spec.N} D={spec.D} C={spec.C} M={spec.M}")
    p = W.make(name)
    N = p.N
    A = torch.from_numpy(p.A).to(dev)
    split, thr = torch.from_numpy(p.split).to(dev), torch.from_numpy(p.thr).to(dev)
    Pd, Bd = torch.from_numpy(p.P).to(dev), torch.from_numpy(p.B).to(dev)
    y = torch.empty((N, spec.M), dtype=torch.float32, device=dev)
    if spec.quantized:
        lut, scale, offset = mdn.build_lut(Pd, Bd)
        call = mdn.prepare_matmul(A, split, thr, lut, scale, offset, y_out=y)
    else:
        lut = mdn.build_lut_f32(Pd, Bd)
        call = mdn.prepare_matmul_f32(A, split, thr, lut, y_out=y)
    # warm-up by time as well as by count: a millisecond-long step runs ~10%
    # slower for the first ~50 ms of sustained work
    n_warm, tw0 = 0, time.perf_counter()
    while n_warm < warmup or time.perf_counter() - tw0 < WARM_SECONDS:
        call()
        n_warm += 1
        if n_warm % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    step_s = e0.elapsed_time(e1) / 1e3 / steps
    y_host = y.cpu().numpy()
    graph_us = None
    if name == "classifier_tiny":
        # back-to-back calls of this layer are bound by the host's enqueue
        # rate: replayed from a captured graph of 20 calls, the step is the
        # kernel's own time
        def gcall():
            mdn.matmul(A, split, thr, lut, scale, offset, y_out=y)
        try:
            gcall()
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for _ in range(20):
                    gcall()
            graph.replay()
            torch.cuda.synchronize()
            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            g0.record()
            for _ in range(10):
                graph.replay()
            g1.record()
            torch.cuda.synchronize()
            graph_us = round(g0.elapsed_time(g1) / 200 * 1e3, 2)
            del graph
        except RuntimeError as exc:   # context only
            graph_us = f"capture failed: {exc}"[:200]
    abytes = algorithmic_bytes(spec, N)
    out = {"N": N, "D": spec.D, "C": spec.C, "M": spec.M, "table": "int8" if spec.quantized else "fp32",
           "rows_per_s": round(N / wall, 1), "step_us": round(step_s * 1e6, 2),
           "wall_us_per_step": round(wall * 1e6, 2), "algorithmic_bytes": abytes,
           "hbm_frac": round(abytes / step_s / 1e9 / HBM_PEAK_GBS, 4), "steps": steps, "warmup": n_warm,
           "a_coverage": a_coverage(p.split, spec.D, spec.D)}
    if graph_us is not None:
        out["graph_step_us"] = graph_us
    if mdn.matmul_index_bytes(A, spec.C, spec.M, f32=not spec.quantized) > 0:
        idx = torch.empty((N, spec.C), dtype=torch.uint8, device=dev)
        enc_us = region_us(lambda i: mdn.encode(A, split, thr, idx_out=idx), stream, reps=10, warm=3)
        if spec.quantized:
            acc_us = region_us(lambda i: mdn.lut_accumulate(idx, lut, scale, offset, y_out=y), stream, reps=10, warm=3)
        else:
            acc_us = region_us(lambda i: mdn.lut_accumulate_f32(idx, lut, y_out=y), stream, reps=10, warm=3)
        out.update({"encode_us": round(enc_us, 2), "accumulate_us": round(acc_us, 2),
                    "encode_hbm_frac": round((4 * spec.D + spec.C) * N / (enc_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
        if onehot_product_route(spec, N):
            # the one-hot int8 product on the matrix cores: N x 16 C x M
            # multiply-adds (dense-equivalent: the kernel issues them as 2:4
            # sparse products) against the dense int8 peak, never the sparse
            # one, and the output stores against the HBM peak
            macs = N * 16 * spec.C * spec.M
            out.update({"accumulate_route": "one-hot int8 product (matrix cores)",
                        "accumulate_mfma_frac": round(2 * macs / (acc_us * 1e-6) / 1e12 / I8_MFMA_PEAK_TOPS, 4),
                        "accumulate_macs": macs,
                        "accumulate_store_hbm_frac": round(4 * N * spec.M / (acc_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
        else:
            lds_bytes = N * spec.C * spec.M * (2 if spec.quantized else 4)
            out.update({"accumulate_route": "gathers from LDS",
                        "accumulate_lds_frac": round(lds_bytes / (acc_us * 1e-6) / 1e12 / LDS_PEAK_TBS, 4),
                        "accumulate_lds_read_bytes": lds_bytes})
        del idx
    torch.backends.cuda.matmul.allow_tf32 = False
    gout = torch.empty((N, spec.M), dtype=torch.float32, device=dev)
    gemm_us = region_us(lambda i: torch.mm(A, Bd, out=gout), stream, reps=5, warm=2)
    out["dense_fp32_gemm_us"] = round(gemm_us, 2)
    del gout, A, y, Pd, Bd, lut
    torch.cuda.empty_cache()
    rows = np.arange(N) if N <= 8192 else sampled_rows(N, sample_n)
    out["parity"] = parity_report(p, y_host, rows)
    if N > 8192:
        out["parity"]["sample"] = f"first and last {sample_n // 4} rows and {sample_n // 2} random rows"
    return out


FIT_TRAIN_ROWS = 16384    # training rows for the table fit (the paper's layers use 10,000)
FIT_HELDOUT_ROWS = 8192
FIT_LAMBDA = 1.0
FIT_GD_STEPS = 10


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--one-core-seconds", type=float, default=3.0)
    ap.add_argument("--workload-steps", type=int, default=10)
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the compact block for the other four workloads")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-context", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="also run a plain device copy of this size (for counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the path would shard by rows with the tables replicated and no exchange (each GPU "
              "running this step on its share); no multi-GPU path is implemented", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2207_05808_amd as mdn
    from paper_2207_05808_amd import workloads as W

    name = args.workload or W.HEADLINE
    spec = W.SPECS[name]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    log(f"[bench] drawing workload {name}: N={spec.N} D={spec.D} C={spec.C} M={spec.M}")
    p = W.make(name)
    N = p.N

    # two copies of A so that consecutive steps never find their input in the
    # 256 MB last-level cache (the headline A is 302 MB)
    A_bufs = [torch.from_numpy(p.A).to(dev) for _ in range(2)]
    split = torch.from_numpy(p.split).to(dev)
    thr = torch.from_numpy(p.thr).to(dev)
    Pd, Bd = torch.from_numpy(p.P).to(dev), torch.from_numpy(p.B).to(dev)
    if spec.quantized:
        lut, scale, offset = mdn.build_lut(Pd, Bd)
    else:
        lut, scale, offset = mdn.build_lut_f32(Pd, Bd), None, None
    y = torch.empty((N, spec.M), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    # arguments marshalled once per input buffer: a step is one C-ABI call
    if spec.quantized:
        calls = [mdn.prepare_matmul(A_bufs[j], split, thr, lut, scale, offset, y_out=y) for j in range(2)]
    else:
        calls = [mdn.prepare_matmul_f32(A_bufs[j], split, thr, lut, y_out=y) for j in range(2)]

    def step(i):
        calls[i % 2]()

    log(f"[bench] warmup {args.warmup} steps")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    K = args.steps
    # one event pair on the launch stream around the K back-to-back launches
    # (the host enqueues far faster than the GPU drains): elapsed / K is the
    # average launch duration, the figure a kernel trace reports
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {K} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(K):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_s = e0.elapsed_time(e1) / 1e3
    ms_per_step = wall / K * 1e3
    avg_kern_s = gpu_s / K
    value = N / (wall / K)
    log(f"[bench] wall {ms_per_step * 1e3:.1f} us/step, kernel avg {avg_kern_s * 1e6:.1f} us")

    # the timed outputs against the oracle: every row of the tiny classifier
    # and of the headline layer, a sample of the larger ones
    y_host = y.cpu().numpy()
    parity = parity_report(p, y_host, np.arange(N) if N <= 200000 else sampled_rows(N))
    del y_host

    # after the timed region: minimum and median over five more repeats of the
    # K launches, and the copy-rate peak
    k_min, k_med = repeat_us(step, stream, K)
    copy_gbs = copy_peak_gbs(dev)

    abytes = algorithmic_bytes(spec, N)
    achieved = abytes / avg_kern_s / 1e9
    kh = kernel_source_hash()
    traffic = stored_traffic(name, kh)
    headline = name == W.HEADLINE
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes": abytes, "kernel_us": round(avg_kern_s * 1e6, 2),
                "kernel_us_min": round(k_min, 2), "kernel_us_median": round(k_med, 2),
                "copy_peak": round(copy_gbs, 1), "frac_of_copy_peak": round(achieved / copy_gbs, 4),
                "a_coverage": a_coverage(p.split, spec.D, spec.D),
                "kernel": ("gfused_kernel<int8> (maddness_matmul, one launch per step)" if headline else
                           "whole step (maddness_matmul%s: encode + accumulate launches)"
                           % ("" if spec.quantized else "_f32")),
                "kernel_source_hash": kh}

    result = {
        "metric": "rows/sec + achieved HBM GB/s (fraction of peak) for fused encode+LUT matmul",
        "value": round(value, 1), "unit": "rows/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32 in / int8 table / int32 accumulate" if spec.quantized else "fp32 in / fp32 table / fp32 accumulate",
        "data": "synthetic",
        "config": {"workload": name, "N": N, "D": spec.D, "C": spec.C, "K": 16, "M": spec.M,
                   "table": "int8 block floating point" if spec.quantized else "fp32",
                   "parallelism": "single GPU"},
        "roofline": roofline,
        "parity": parity,
    }

    if not args.no_context:
        # the two steps as separate calls (encode to an index buffer, then the
        # accumulate-only entry point), same region timing as the fused step
        idx = torch.empty((N, spec.C), dtype=torch.uint8, device=dev)
        split_calls = [lambda j=j: mdn.encode(A_bufs[j], split, thr, idx_out=idx, validate=False) for j in range(2)]
        if spec.quantized:
            acc_call = lambda: mdn.lut_accumulate(idx, lut, scale, offset, y_out=y, validate=False)
        else:
            acc_call = lambda: mdn.lut_accumulate_f32(idx, lut, y_out=y)

        _region = region_us
        region_us_ = lambda fn, reps=20: _region(fn, stream, reps=reps)   # noqa: E731

        enc_us = region_us_(lambda i: split_calls[i % 2]())
        acc_us = region_us_(lambda i: acc_call())
        result["context"] = {"encode_only_us": round(enc_us, 2), "accumulate_only_us": round(acc_us, 2)}
        if not headline and onehot_product_route(spec, N):
            # the one-hot int8 product on the matrix cores: N x 16 C x M
            # multiply-adds (dense-equivalent, issued as 2:4 sparse products)
            # against the dense int8 peak
            macs = N * 16 * spec.C * spec.M
            tops = 2 * macs / (acc_us * 1e-6) / 1e12
            result["context"]["accumulate_mfma_roofline"] = {
                "bound": "mfma", "achieved": round(tops, 1), "peak": I8_MFMA_PEAK_TOPS, "unit": "TOP/s",
                "frac": round(tops / I8_MFMA_PEAK_TOPS, 4), "macs": macs}
        elif not headline:
            # the accumulate of the other two-phase workloads is bound by LDS
            # reads: N C M lookups of 2 bytes (int8 tables, staged as 16-bit
            # entries) or 4 bytes (fp32), against 256 B/clk/CU x 256 CUs x
            # 2.4 GHz
            lds_bytes = N * spec.C * spec.M * (2 if spec.quantized else 4)
            lds_tbps = lds_bytes / (acc_us * 1e-6) / 1e12
            result["context"]["accumulate_lds_roofline"] = {
                "bound": "lds", "achieved": round(lds_tbps, 2), "peak": LDS_PEAK_TBS, "unit": "TB/s",
                "frac": round(lds_tbps / LDS_PEAK_TBS, 4), "lds_read_bytes": lds_bytes}
        if spec.quantized:
            # the rounded 8-bit averaging accumulate (approximate) over a
            # shared-exponent table of the same weights, on the same indices
            slut, sscale, soffset = mdn.build_lut_shared(Pd, Bd)
            avg_us = region_us_(lambda i: mdn.lut_accumulate_avg(idx, slut, sscale, soffset, y_out=y))
            result["context"]["accumulate_avg8_us"] = round(avg_us, 2)
            # its accuracy cost: relative Frobenius distance to the exact sum
            # over the same shared-exponent table
            _, y_exact = mdn.lut_accumulate(idx, slut, sscale, soffset)
            torch.cuda.synchronize()
            dd = y.double() - y_exact.double()
            ref = y_exact.double().norm()
            result["context"]["avg8_rel_frobenius_diff"] = float(f"{float(dd.norm() / ref):.4g}")
            # the same with the mean difference (the rounding's upward bias) taken out
            result["context"]["avg8_rel_frobenius_diff_centered"] = float(f"{float((dd - dd.mean()).norm() / ref):.4g}")
            del dd
            del slut, y_exact
        del idx
        # the same step with the layer output sigma fused (bias + ReLU, bias + row softmax)
        cb = torch.from_numpy(np.random.default_rng(1).standard_normal(spec.M).astype(np.float32)).to(dev)
        for act in ("relu", "softmax"):
            if spec.quantized:
                f = lambda i, a=act: mdn.matmul_act(A_bufs[i % 2], split, thr, lut, scale, offset, col_bias=cb,
                                                    act=a, y_out=y)
            else:
                f = lambda i, a=act: mdn.matmul_act_f32(A_bufs[i % 2], split, thr, lut, col_bias=cb, act=a, y_out=y)
            result["context"][f"step_with_{act}_us"] = round(region_us_(f), 2)

        # the same step replayed from a captured HIP graph of 20 steps, as a
        # serving loop that captures its launches runs it (launch-bound
        # layers gain); two-phase workloads get a caller index buffer, so the
        # captured calls allocate nothing
        gidx = None if headline or name == "classifier_tiny" else torch.empty((N, spec.C), dtype=torch.uint8, device=dev)

        def graph_step(i):
            if spec.quantized:
                mdn.matmul(A_bufs[i % 2], split, thr, lut, scale, offset, y_out=y, idx_out=gidx)
            else:
                mdn.matmul_f32(A_bufs[i % 2], split, thr, lut, y_out=y, idx_out=gidx)

        try:
            for i in range(2):
                graph_step(i)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            gsteps = 20
            with torch.cuda.graph(graph):
                for i in range(gsteps):
                    graph_step(i)
            graph.replay()
            torch.cuda.synchronize()
            gr0, gr1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            greps = 5
            gr0.record()
            for _ in range(greps):
                graph.replay()
            gr1.record()
            torch.cuda.synchronize()
            result["context"]["graph_step_us"] = round(gr0.elapsed_time(gr1) / (greps * gsteps) * 1e3, 2)
            del graph
        except RuntimeError as exc:   # context only: the bench line does not depend on it
            result["context"]["graph_step_us"] = f"capture failed: {exc}"[:200]
        del gidx

        # dense fp32 GEMM of the same shape (torch -> hipBLASLt / rocBLAS), TF32 off
        torch.backends.cuda.matmul.allow_tf32 = False
        out = torch.empty((N, spec.M), dtype=torch.float32, device=dev)
        for _ in range(3):
            torch.mm(A_bufs[0], Bd, out=out)
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 10
        g0.record()
        for i in range(reps):
            torch.mm(A_bufs[i % 2], Bd, out=out)
        g1.record()
        torch.cuda.synchronize()
        gms = g0.elapsed_time(g1) / reps
        result["context"].update({"dense_fp32_gemm_us": round(gms * 1e3, 2),
                                  "dense_fp32_gemm_tflops": round(2.0 * N * spec.D * spec.M / (gms / 1e3) / 1e12, 2),
                                  "fused_speedup_vs_gemm": round(gms / 1e3 / avg_kern_s, 3)})
        del out

        # offline table construction on the GPU: T = P B in double, then the
        # 8-bit block floating point quantizer (or the fp32 rounding)
        if spec.quantized:
            build_us = region_us_(lambda i: mdn.build_lut(Pd, Bd), reps=3)
        else:
            build_us = region_us_(lambda i: mdn.build_lut_f32(Pd, Bd), reps=3)
        result["context"]["build_lut_ms"] = round(build_us / 1e3, 3)

        # model-aware table fit (Eq. 3, affine output) on 16384 training rows
        # of the same layer (targets Y = AB, prototype table T0 = P B), and
        # its effect on 8192 held-out rows through the fp32-table accumulate
        n_tr = min(N // 2, FIT_TRAIN_ROWS)
        n_ho = min(N - n_tr, FIT_HELDOUT_ROWS)
        A_tr, A_ho = A_bufs[0][:n_tr], A_bufs[0][n_tr:n_tr + n_ho]
        Y_tr, Y_ho = torch.mm(A_tr, Bd), torch.mm(A_ho, Bd)
        idx_tr, idx_ho = mdn.encode(A_tr, split, thr), mdn.encode(A_ho, split, thr)
        T0 = mdn.build_lut_f32(Pd, Bd)
        ws = torch.empty((mdn.fit_lut_workspace_bytes(n_tr, spec.C) + 256,), dtype=torch.uint8, device=dev)
        fit_us = region_us_(lambda i: mdn.fit_lut_ridge(idx_tr, Y_tr, T0, FIT_LAMBDA, workspace=ws), reps=3)
        T_fit = mdn.fit_lut_ridge(idx_tr, Y_tr, T0, FIT_LAMBDA, workspace=ws).float()

        def rel_err(T):
            yh = mdn.lut_accumulate_f32(idx_ho, T)
            torch.cuda.synchronize()
            return float((yh.double() - Y_ho.double()).norm() / Y_ho.double().norm())

        # the nonlinear objectives (ReLU + squared error, softmax + KL
        # divergence) by gradient descent: time per step over 10 steps, step
        # 1 / (2 C Nb + 2 lambda) (Nb the largest bucket: Gershgorin bound on
        # the curvature)
        nb_max = max(int(torch.bincount(idx_tr[:, c].long(), minlength=16).max()) for c in range(spec.C))
        eta = 1.0 / (2.0 * spec.C * nb_max + 2.0 * FIT_LAMBDA)
        ws_gd = torch.empty((mdn.fit_lut_gd_workspace_bytes(n_tr, spec.C, spec.M) + 256,), dtype=torch.uint8,
                            device=dev)
        for act in ("relu", "softmax"):
            us = region_us_(lambda i, a=act: mdn.fit_lut_gd(idx_tr, Y_tr, T0, a, FIT_LAMBDA, eta, FIT_GD_STEPS,
                                                            workspace=ws_gd), reps=2)
            result["context"][f"fit_gd_{act}_ms_per_step"] = round(us / 1e3 / FIT_GD_STEPS, 3)
        del ws_gd
        result["context"].update({"fit_lut_ridge_ms": round(fit_us / 1e3, 3), "fit_train_rows": n_tr,
                                  "fit_lambda": FIT_LAMBDA,
                                  "heldout_rel_err_prototype_table": float(f"{rel_err(T0):.4g}"),
                                  "heldout_rel_err_fitted_table": float(f"{rel_err(T_fit):.4g}")})
        del ws, T0, T_fit, Y_tr, Y_ho, idx_tr, idx_ho
    del Pd

    if args.copy_calibration_mb > 0:
        nb = args.copy_calibration_mb << 20
        src = torch.ones(nb // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):   # device-to-device copies: the runtime's plain copy kernel
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: 3 x ({nb} bytes read + {nb} bytes written)")

    if not args.no_context and not args.no_workloads and args.workload is None:
        del A_bufs, y, calls, lut, scale, offset
        torch.cuda.empty_cache()
        result["context"]["workloads"] = {
            w: workload_block(w, args.workload_steps, 3) for w in W.SPECS if w != W.HEADLINE}

    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle baseline (~{args.cpu_seconds:.0f} s + {args.one_core_seconds:.0f} s on one core)")
        result["cpu_baseline"] = cpu_baseline(p, args.cpu_seconds, args.one_core_seconds)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
