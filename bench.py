#!/usr/bin/env python3
"""Benchmark for integer GEMM C += A.B on one MI355X.

A step is one call of igemm_i16 on the int16 workload m = n = k = 4096
(A, B uniform over the full int16 range, C uniform in [-2^20, 2^20], seed 1):
host validation and planning, the two pack kernels (A split into int8 limb
planes with its row sums, B transposed and split with its column sums, into
a workspace from torch's caching allocator), then the multiply kernel that
streams the packed planes through LDS into the int8 matrix cores, applies
the limb corrections and adds into C with int32 wraparound. Inputs are
resident in HBM before the timed region starts.

Prints ONE JSON line. Besides the headline value it carries:
  roofline      the dominant kernel (the multiply) timed alone with HIP events
                on the stream it is launched on, by running it on operands
                packed once (the library's pack-once calls), against the
                int8 matrix-core peak divided by the four limb products,
                with the matrix-core utilisation, int8 operations and clock
                rocprofv3 counted for that kernel (committed summary);
  cpu_baseline  the CPU oracle timed on the host cores over a bounded sample
                of the same workload;
  per_config    every other workload, each by graph replay (median of five
                repetitions of at least 20 ms; memory-bound ones rotate
                through enough buffer sets to defeat the 256 MB last-level
                cache), with its own roofline fraction (memory-bound ones
                also against a measured 1 GiB device copy); then the
                paper's own GEMM shape (4096, 4096, 290), for context, the
                same shape through the int16-output entry point with the
                paper's k_c = 290 and shift 0 (and 4096^3 with k_c = 256),
                and the six network layers run as convolutions through the
                implicit-GEMM entry point (IM2ROW gathered in the kernel), at
                batch 1 and batch 32.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-extra]
                       [--no-cpu-baseline] [--cpu-seconds S]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published dense peaks and bandwidth.
PEAK_INT8_TOPS = 5000.0      # int8 MFMA, dense
HBM_GBS = 8000.0             # HBM3E
LIMB_PRODUCTS_I16 = 4        # int8 products per int16 multiply-add
PEAK_I16_TOPS = PEAK_INT8_TOPS / LIMB_PRODUCTS_I16
MALL_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_i16_packed_128x128_4096cube.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2302_07594_amd", "csrc", "igemm_packed.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return t.get("traffic_bytes_per_launch")


MFMA_FILES = {
    "i16": os.path.join(ROOT, "profiles", "mfma_i16_packed_128x128_4096cube.json"),
    "i8": os.path.join(ROOT, "profiles", "mfma_i8_packed_256x256_8192cube.json"),
}


def measured_mfma(dtype):
    """Matrix-core figures of the packed multiply from the committed
    rocprofv3 counter summary (SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_I8,
    GRBM_GUI_ACTIVE with a kernel trace), if taken on the current kernel
    source; otherwise None."""
    try:
        with open(MFMA_FILES[dtype]) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash() or not t.get("dispatches"):
        return None
    rows = t["dispatches"]
    avg = lambda key: sum(r[key] for r in rows) / len(rows)
    return {
        "mfma_busy": round(avg("mfma_busy"), 4),
        "int8_mfma_ops_per_launch": rows[0]["int8_mfma_ops"],
        "clock_ghz": round(avg("clock_ghz"), 3),
        "dispatches": len(rows),
        "source": os.path.relpath(MFMA_FILES[dtype], ROOT),
    }


def roofline_for(dtype, m, n, k, seconds):
    """(bound, achieved, peak, unit) for one GEMM of this shape."""
    es = 2 if dtype == "i16" else 1
    ops = 2.0 * m * n * k
    nbytes = m * k * es + k * n * es + 8.0 * m * n
    peak_ops = (PEAK_I16_TOPS if es == 2 else PEAK_INT8_TOPS) * 1e12
    if ops / nbytes >= peak_ops / (HBM_GBS * 1e9):
        return "mfma", ops / seconds / 1e12, peak_ops / 1e12, "TOPS"
    return "hbm", nbytes / seconds / 1e9, HBM_GBS, "GB/s"


def time_graph(g, per_graph, reps=5, min_rep_ms=20.0):
    """Device time per launch of a captured graph of per_graph launches: the
    median over `reps` repetitions, each replaying the graph back to back for
    at least min_rep_ms (HIP events on the current stream)."""
    import statistics

    import torch
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    per_replay_ms = max(e0.elapsed_time(e1), 1e-3)
    n = max(1, -(-int(min_rep_ms * 1000) // int(per_replay_ms * 1000 + 1)))
    times = []
    for _ in range(reps):
        e0.record()
        for _ in range(n):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3 / (n * per_graph))
    return statistics.median(times)


TIMING = "hip graph replay: median of 5 repetitions of >= 20 ms"


def copy_bandwidth(nbytes=1 << 30, reps=5):
    """Device-to-device copy rate (bytes read plus written per second) of a
    1 GiB buffer, larger than the 256 MB last-level cache."""
    import statistics

    import torch
    x = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    for _ in range(2):
        y.copy_(x)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        y.copy_(x)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    del x, y
    torch.cuda.empty_cache()
    return 2.0 * nbytes / statistics.median(ts)


def bench_case(case, min_sets=1, per_graph=40, warmup=3):
    """Time one workload case on rotating device copies of its operands.

    The launches are captured once in a HIP graph (per_graph launches cycling
    through the buffer sets) and the graph is replayed, so the figure is the
    device time per launch without host launch overhead.
    """
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    A, B, C = workloads.generate(case)
    es = 2 if case.dtype == "i16" else 1
    set_bytes = A.nbytes + B.nbytes + C.nbytes
    nsets = max(min_sets, -(-2 * MALL_BYTES // set_bytes))
    nsets = min(nsets, 64)
    Ad0, Bd0, Cd0 = (torch.from_numpy(x).cuda() for x in (A, B, C))
    sets = [(Ad0, Bd0, Cd0)] + [(Ad0.clone(), Bd0.clone(), Cd0.clone()) for _ in range(nsets - 1)]
    f = ig.gemm_i16 if es == 2 else ig.gemm_i8
    for i in range(warmup):
        f(*sets[i % nsets])
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            f(*sets[i % nsets])
    g.replay()
    torch.cuda.synchronize()
    t = time_graph(g, per_graph)
    plan = ig.igemm_query_plan(es, case.m, case.n, case.k)
    bound, ach, peak, unit = roofline_for(case.dtype, case.m, case.n, case.k, t)
    return {
        "name": case.name, "dtype": case.dtype, "m": case.m, "n": case.n, "k": case.k,
        "kernel": plan["kernel_name"], "split": plan["split"], "grid": plan["grid"],
        "us": round(t * 1e6, 2), "TOPS": round(2.0 * case.m * case.n * case.k / t / 1e12, 2),
        "bound": bound, "achieved": round(ach, 1), "peak": peak, "unit": unit,
        "frac": round(ach / peak, 4), "buffer_sets": nsets, "timing": TIMING,
        # the int8 counter summary was taken on this very workload
        **({"rocprof_mfma": measured_mfma("i8")}
           if (case.dtype, case.m, case.n, case.k) == ("i8", 8192, 8192, 8192) else {}),
    }


def bench_srs_case(case, kc, shift, per_graph=40, warmup=3):
    """Time the int16-output update (shift-round-saturate conversion per k
    block of kc, int16 C) on a workload's A and B with a random int16 C, like
    bench_case: gemm_srs as a caller gets it, i.e. the packed path (operands
    packed into a workspace from torch's allocator, one multiply per block)
    where the library chooses it, else one fused launch per block. The
    algorithmic bytes are A and B once and the int16 C read and written once
    per block."""
    import numpy as np
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    A, B, _ = workloads.generate(case)
    C = np.random.default_rng(case.seed).integers(-32768, 32767, size=(case.m, case.n),
                                                  dtype=np.int16, endpoint=True)
    set_bytes = A.nbytes + B.nbytes + C.nbytes
    nsets = min(64, max(1, -(-2 * MALL_BYTES // set_bytes)))
    Ad0, Bd0, Cd0 = (torch.from_numpy(x).cuda() for x in (A, B, C))
    sets = [(Ad0, Bd0, Cd0)] + [(Ad0.clone(), Bd0.clone(), Cd0.clone()) for _ in range(nsets - 1)]
    for i in range(warmup):
        ig.gemm_srs(*sets[i % nsets], kc=kc, shift=shift)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            ig.gemm_srs(*sets[i % nsets], kc=kc, shift=shift)
    g.replay()
    torch.cuda.synchronize()
    t = time_graph(g, per_graph)
    m, n, k = case.m, case.n, case.k
    nblocks = 1 if (kc == 0 or kc >= k) else -(-k // kc)
    ws_bytes = ig.igemm_srs_query(2 if case.dtype == "i16" else 1, m, n, k, Ad0, k, Bd0, n, Cd0,
                                  n, kc, torch.cuda.get_device_properties(0).multi_processor_count)
    ops = 2.0 * m * n * k
    nbytes = A.nbytes + B.nbytes + 4.0 * m * n * nblocks
    peak_ops = PEAK_I16_TOPS * 1e12
    if ops / nbytes >= peak_ops / (HBM_GBS * 1e9):
        bound, ach, peak, unit = "mfma", ops / t / 1e12, peak_ops / 1e12, "TOPS"
    else:
        bound, ach, peak, unit = "hbm", nbytes / t / 1e9, HBM_GBS, "GB/s"
    return {
        "name": f"{case.name}_srs_kc{kc}_shift{shift}", "dtype": case.dtype,
        "m": m, "n": n, "k": k, "kc": kc, "shift": shift, "blocks": nblocks,
        "epilogue": "int16 C += sat16(floor(block product / 2^shift)) modulo 2^16",
        "path": "packed" if ws_bytes > 0 else "fused", "workspace_bytes": ws_bytes,
        "us": round(t * 1e6, 2), "TOPS": round(ops / t / 1e12, 2),
        "bound": bound, "achieved": round(ach, 1), "peak": peak, "unit": unit,
        "frac": round(ach / peak, 4), "buffer_sets": nsets, "timing": TIMING,
    }


def bench_conv_case(case, per_graph=40, warmup=3):
    """Time one convolution (implicit GEMM: IM2ROW gathered in the kernel)
    like bench_case; the roofline counts the lowered GEMM's multiply-adds
    and the unique bytes of X, W and Y (read and written)."""
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    X, W, Y = workloads.generate_conv(case)
    es = 2 if case.dtype == "i16" else 1
    set_bytes = X.nbytes + W.nbytes + Y.nbytes
    nsets = min(64, max(1, -(-2 * MALL_BYTES // set_bytes)))
    Xd0, Wd0, Yd0 = (torch.from_numpy(x).cuda() for x in (X, W, Y))
    sets = [(Xd0, Wd0, Yd0)] + [(Xd0.clone(), Wd0.clone(), Yd0.clone()) for _ in range(nsets - 1)]
    kw = dict(stride=case.stride, pad=case.pad, dil=case.dil)
    for i in range(warmup):
        ig.conv2d(*sets[i % nsets], **kw)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            ig.conv2d(*sets[i % nsets], **kw)
    g.replay()
    torch.cuda.synchronize()
    t = time_graph(g, per_graph)
    m, n, k = case.gemm_shape()
    d = ig.conv_desc(case.n, case.h, case.w, case.c, case.k, case.r, case.s, case.stride,
                     case.pad, case.dil)
    plan = ig.igemm_conv2d_query_plan(es, d, Xd0, Wd0, Yd0)
    ops = 2.0 * m * n * k
    nbytes = X.nbytes + W.nbytes + 2.0 * Y.nbytes
    peak_ops = (PEAK_I16_TOPS if es == 2 else PEAK_INT8_TOPS) * 1e12
    if ops / nbytes >= peak_ops / (HBM_GBS * 1e9):
        bound, ach, peak, unit = "mfma", ops / t / 1e12, peak_ops / 1e12, "TOPS"
    else:
        bound, ach, peak, unit = "hbm", nbytes / t / 1e9, HBM_GBS, "GB/s"
    return {
        "name": case.name, "dtype": case.dtype, "conv": {
            "n": case.n, "h": case.h, "w": case.w, "c": case.c, "k": case.k, "r": case.r,
            "s": case.s, "stride": list(case.stride), "pad": list(case.pad),
            "dil": list(case.dil)},
        "m": m, "n": n, "k": k, "kernel": plan["kernel_name"], "split": plan["split"],
        "grid": plan["grid"], "vector_gather": bool(plan["vec_a"]),
        "us": round(t * 1e6, 2), "TOPS": round(ops / t / 1e12, 2),
        "bound": bound, "achieved": round(ach, 1), "peak": peak, "unit": unit,
        "frac": round(ach / peak, 4), "buffer_sets": nsets, "timing": TIMING,
    }


def cpu_baseline(A, B, C_gpu_first, C0, seconds):
    """Time the CPU oracle on whole rows of the same workload, for at most
    about `seconds`; also confirm those rows match the GPU's first result."""
    import numpy as np

    import oracle
    m, k = A.shape
    n = B.shape[1]
    block = 64
    done = 0
    elapsed = 0.0
    mismatched = 0
    while done < m and elapsed < seconds:
        rows = slice(done, min(m, done + block))
        Cr = np.ascontiguousarray(C0[rows])
        t0 = time.perf_counter()
        oracle.igemm(np.ascontiguousarray(A[rows]), B, Cr)
        elapsed += time.perf_counter() - t0
        mismatched += int((Cr != C_gpu_first[rows]).sum())
        done = rows.stop
    ops = 2.0 * done * n * k
    return {
        "value": round(ops / elapsed / 1e12, 6), "unit": "TOPS",
        "cores": oracle.num_threads(), "kind": "oracle",
        "sample": f"rows 0..{done - 1} of the {m}x{n}x{k} int16 workload "
                  f"({done * n * k:.3g} multiply-adds, {elapsed:.1f} s)",
        "rows_bit_exact_vs_gpu": mismatched == 0, "rows_checked": done,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-extra", action="store_true", help="skip the per-config table")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the benchmark measures one GPU "
              "(the kernel at one GPU's share); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2302_07594_amd as ig
    import workloads

    case = workloads.WORKLOADS["i16_4096"].cases[0]
    m, n, k = case.m, case.n, case.k
    log(f"bench: generating {case.name}")
    A, B, C0 = workloads.generate(case)
    Ad = torch.from_numpy(A).cuda()
    Bd = torch.from_numpy(B).cuda()
    Cd = torch.from_numpy(C0).cuda()
    # First launch on the pristine C; its result is compared with the oracle
    # rows in the CPU-baseline leg.
    ig.gemm_i16(Ad, Bd, Cd)
    torch.cuda.synchronize()
    C_first = Cd.cpu().numpy()
    plan = ig.igemm_query_plan(2, m, n, k, Ad, k, Bd, n, Cd, n)

    log(f"bench: warmup {args.warmup}, timed steps {args.steps}")
    for _ in range(args.warmup):
        ig.gemm_i16(Ad, Bd, Cd)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        ig.gemm_i16(Ad, Bd, Cd)
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = (t1 - t0) / args.steps
    step_dev = e0.elapsed_time(e1) * 1e-3 / args.steps
    ops = 2.0 * m * n * k
    value = ops / wall / 1e12

    # The dominant kernel alone: the multiply on operands packed once. Its
    # launches go to the current stream, where the events are recorded.
    log("bench: multiply kernel alone on packed operands")
    P = ig.pack(Ad, Bd)
    Cm = Cd.clone()
    for _ in range(3):
        ig.gemm_prepacked(P, Cm)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        ig.gemm_prepacked(P, Cm)
    e1.record()
    torch.cuda.synchronize()
    mult = e0.elapsed_time(e1) * 1e-3 / args.steps
    e0.record()
    for _ in range(args.steps):
        ig.igemm_pack_i16(m, n, k, Ad, k, Bd, n, P.kernel, P.workspace, P.nbytes)
    e1.record()
    torch.cuda.synchronize()
    pack_t = e0.elapsed_time(e1) * 1e-3 / args.steps
    del P, Cm
    ach = ops / mult / 1e12

    out = {
        "metric": "int16 GEMM C+=A.B throughput on 1 MI355X (int8 MFMA limb split), TOPS",
        "value": round(value, 2), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int16", "data": "synthetic",
        "config": {
            "workload": "int16 GEMM C += A.B, m=n=k=4096, row-major, A,B uniform over the full "
                        "int16 range, C uniform in [-2^20,2^20], int32 wraparound, seed 1",
            "m": m, "n": n, "k": k, "accumulate": "int32 modulo 2^32",
            "kernel": plan["kernel_name"], "split": plan["split"], "grid": plan["grid"],
            "workspace_bytes": plan["workspace_bytes"],
        },
        "roofline": {
            "bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_I16_TOPS, "unit": "TOPS",
            "frac": round(ach / PEAK_I16_TOPS, 4), "traffic": measured_traffic(),
            "kernel": "igemm_packed<int16, 128x128> (multiply on packed operands)",
            "peak_basis": "int8 MFMA dense peak 5000 TOPS / 4 int8 limb products per int16 "
                          "multiply-add",
            "int8_mfma_frac": round(ach * LIMB_PRODUCTS_I16 / PEAK_INT8_TOPS, 4),
            "kernel_us": round(mult * 1e6, 2),
            "pack_us": round(pack_t * 1e6, 2),
            "step_device_us": round(step_dev * 1e6, 2),
            "rocprof_mfma": measured_mfma("i16"),
        },
    }
    if not args.no_cpu_baseline:
        log("bench: CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(A, B, C_first, C0, args.cpu_seconds)
    del Ad, Bd, Cd
    torch.cuda.empty_cache()
    if not args.no_extra:
        per = []
        for wname in ("i16_256", "i8_8192", "i16_conv", "i8_skinny", "i16_paper"):
            for c in workloads.WORKLOADS[wname].cases:
                log(f"bench: per-config {c.name}")
                per.append(bench_case(c))
                torch.cuda.empty_cache()
        # The paper's configuration: its GEMM shape with its k_c = 290 and the
        # listing's shift 0, int16 output; and 4096^3 with k_c = 256.
        log("bench: per-config int16-output update")
        per.append(bench_srs_case(workloads.WORKLOADS["i16_paper"].cases[0], 290, 0))
        per.append(bench_srs_case(workloads.WORKLOADS["i16_4096"].cases[0], 256, 0,
                                  per_graph=10))
        torch.cuda.empty_cache()
        for c in workloads.CONV2D_CASES + workloads.CONV2D_B32_CASES:
            log(f"bench: per-config {c.name}")
            per.append(bench_conv_case(c, per_graph=40 if c.n == 1 else 10))
            torch.cuda.empty_cache()
        # Memory-bound entries also against a measured device copy.
        log("bench: device-to-device copy bandwidth")
        cbw = copy_bandwidth()
        out["copy_bandwidth_GBs"] = round(cbw / 1e9, 1)
        for r in per:
            if r["bound"] == "hbm":
                r["frac_of_copy"] = round(r["achieved"] * 1e9 / cbw, 4)
        out["per_config"] = per
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
