#!/usr/bin/env python3
"""Benchmark for integer GEMM C += A.B on one MI355X.

A step is one call of igemm_i16 on the int16 workload m = n = k = 4096
(A, B uniform over the full int16 range, C uniform in [-2^20, 2^20], seed 1)
through the tensor wrapper gemm_i16: host validation and planning, the two
pack kernels (A split into int8 limb planes with its row sums, B transposed
and split with its column sums, into a workspace from torch's caching
allocator), then the multiply kernel that streams the packed planes through
LDS into the int8 matrix cores, applies the limb corrections and adds into C
with int32 wraparound. Inputs are resident in HBM before the timed region
starts.

Prints ONE JSON line. Besides the headline value it carries:
  roofline      the dominant kernel (the multiply) timed alone with HIP events
                on the stream it is launched on, by running it on operands
                packed once (the library's pack-once calls), against the
                int8 matrix-core peak divided by the four limb products; the
                whole step's fraction of the same peak beside it; the HBM
                traffic and matrix-core utilisation rocprofv3 counted for that
                kernel (committed summaries, reported while the kernel's
                sources and build flags hash to the value they were taken on);
  cpu_baseline  the CPU oracle on the host cores: its rate on the whole int16
                4096^3 workload, the seconds it took on every other workload
                (each one's first GPU result is compared with it element by
                element), one-thread seconds for int16 256^3, the CPU model;
  per_config    every workload by graph replay (median of five repetitions of
                at least 20 ms), in a compact map name -> {us, TOPS, GB/s for
                memory-bound entries, bound, frac of that roofline, frac of a
                measured 1 GiB device copy, kernel/split, MB cycled per graph
                replay (memory-bound entries rotate at least 512 MB of
                distinct buffers, twice the 256 MB last-level cache), exact =
                the first result equals the oracle's in every element}: int16
                256^3, int8 8192^3, the six conv-shaped int16 GEMMs, the six
                skinny int8 GEMMs, the paper's GEMM shape (4096, 4096, 290)
                for context, the int16-output update on that shape with the
                paper's k_c = 290 and shift 0 and on 4096^3 with k_c = 256,
                and the six network layers as convolutions through the
                implicit-GEMM entry point at batch 1 and batch 32.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-extra]
                       [--no-cpu-baseline] [--details FILE]
"""
from __future__ import annotations

import argparse
import json
import os
import subprocess
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
MIN_CYCLED = 2 * MALL_BYTES  # bytes a memory-bound graph replay must rotate through
# Committed rocprofv3 counter summaries (paper_2302_07594_amd/profile_run.py
# traffic / mfma), per kernel family: (family whose source hash they carry,
# traffic file, matrix-core file).
SUMMARIES = {
    "i16": ("packed", os.path.join(ROOT, "profiles", "traffic_i16_packed_128x128_4096cube.json"),
            os.path.join(ROOT, "profiles", "mfma_i16_packed_128x128_4096cube.json")),
    "i8": ("direct", os.path.join(ROOT, "profiles", "traffic_i8_direct_256x256_8192cube.json"),
           os.path.join(ROOT, "profiles", "mfma_i8_direct_256x256_8192cube.json")),
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash(family) -> str:
    """SHA-256 over a kernel family's sources, the headers they include and
    the library's compile flags."""
    from paper_2302_07594_amd import build as hip_build
    return hip_build.kernel_hash(family)


def _summary(path, family):
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    return t if t.get("kernel_source_sha256") == kernel_source_hash(family) else None


def measured_traffic(dtype):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel sources and flags; otherwise None."""
    family, path, _ = SUMMARIES[dtype]
    t = _summary(path, family)
    return None if t is None else t.get("traffic_bytes_per_launch")


def measured_mfma(dtype):
    """Matrix-core figures of the multiply kernel from the committed
    rocprofv3 counter summary (SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_I8,
    GRBM_GUI_ACTIVE with a kernel trace), if taken on the current kernel
    sources and flags; otherwise None."""
    family, _, path = SUMMARIES[dtype]
    t = _summary(path, family)
    if t is None or not t.get("dispatches"):
        return None
    rows = t["dispatches"]
    avg = lambda key: sum(r[key] for r in rows) / len(rows)
    return {
        "mfma_busy": round(avg("mfma_busy"), 4),
        "int8_mfma_ops_per_launch": rows[0]["int8_mfma_ops"],
        "clock_ghz": round(avg("clock_ghz"), 3),
        "source": os.path.relpath(path, ROOT),
    }


def roofline(ops, nbytes, es, seconds):
    """(bound, achieved, peak, unit) for `ops` operations moving `nbytes`."""
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


class OracleLog:
    """Seconds the CPU oracle took per workload (each check is one whole
    workload, all host threads)."""

    def __init__(self):
        self.seconds = {}

    def run(self, name, fn, *args):
        t0 = time.perf_counter()
        fn(*args)
        self.seconds[name] = round(time.perf_counter() - t0, 3)


def replay_sets(f, host_sets, set_bytes, memory_bound, min_per_graph=40, warmup=3):
    """Capture launches of f over rotating device copies of the operands and
    time the graph. Memory-bound workloads rotate through enough distinct
    buffer sets that one replay touches at least MIN_CYCLED bytes, with at
    least one launch per set, so no launch finds its operands in the
    last-level cache from the launch before. Returns (seconds per launch,
    number of sets, bytes cycled per replay)."""
    import torch
    nsets = -(-MIN_CYCLED // set_bytes) if memory_bound else max(1, -(-MIN_CYCLED // set_bytes))
    if not memory_bound:
        nsets = min(nsets, 2)
    first = [torch.from_numpy(x).cuda() for x in host_sets]
    sets = [first] + [[t.clone() for t in first] for _ in range(nsets - 1)]
    per_graph = max(min_per_graph, nsets)
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
    del g, sets, first
    torch.cuda.empty_cache()
    return t, nsets, min(nsets, per_graph) * set_bytes


def entry(t, ops, nbytes, es, kernel, cycled, exact):
    bound, ach, peak, _ = roofline(ops, nbytes, es, t)
    e = {"us": round(t * 1e6, 2), "TOPS": round(ops / t / 1e12, 2)}
    if bound == "hbm":
        e["GBs"] = round(ach, 1)
    e.update({"bound": bound, "frac": round(ach / peak, 4), "kern": kernel,
              "MB": round(cycled / 1e6), "exact": exact})
    return e


def first_result(f, host):
    """One call on pristine device copies; returns the host result."""
    import torch
    dev = [torch.from_numpy(x).cuda() for x in host]
    f(*dev)
    torch.cuda.synchronize()
    out = dev[-1].cpu().numpy()
    del dev
    return out


def bench_gemm(case, olog, details):
    import numpy as np

    import oracle
    import paper_2302_07594_amd as ig
    import workloads
    A, B, C = workloads.generate(case)
    es = 2 if case.dtype == "i16" else 1
    f = ig.gemm_i16 if es == 2 else ig.gemm_i8
    got = first_result(f, (A, B, C))
    want = C.copy()
    olog.run(case.name, oracle.igemm, A, B, want)
    exact = bool(np.array_equal(got, want))
    del got, want
    m, n, k = case.m, case.n, case.k
    ops = 2.0 * m * n * k
    nbytes = A.nbytes + B.nbytes + 2.0 * C.nbytes
    memory_bound = roofline(ops, nbytes, es, 1.0)[0] == "hbm"
    t, nsets, cycled = replay_sets(f, (A, B, C), A.nbytes + B.nbytes + C.nbytes, memory_bound)
    plan = ig.igemm_query_plan(es, m, n, k)
    e = entry(t, ops, nbytes, es, f"{plan['kernel_name']}/{plan['split']}", cycled, exact)
    if (case.dtype, m, n, k) == ("i8", 8192, 8192, 8192):
        mf = measured_mfma("i8")
        if mf is not None:
            e["mfma_busy"], e["clk_ghz"] = mf["mfma_busy"], mf["clock_ghz"]
        tr = measured_traffic("i8")
        if tr is not None:
            e["hbm_MB"] = round(tr / 1e6, 1)   # counter-measured bytes per launch
    details.append({"name": case.name, "m": m, "n": n, "k": k, "plan": plan, "sets": nsets,
                    **e})
    return e


def bench_srs(case, kc, shift, olog, details):
    """The int16-output update (shift-round-saturate conversion per k block of
    kc, int16 C) on a workload's A and B with a random int16 C, through
    gemm_srs (the packed path on a workspace from torch's allocator where the
    library plans it, else one fused launch per block). Algorithmic bytes: A
    and B once and the int16 C read and written once per block."""
    import numpy as np

    import oracle
    import paper_2302_07594_amd as ig
    import workloads
    A, B, _ = workloads.generate(case)
    C = np.random.default_rng(case.seed).integers(-32768, 32767, size=(case.m, case.n),
                                                  dtype=np.int16, endpoint=True)
    f = lambda a, b, c: ig.gemm_srs(a, b, c, kc=kc, shift=shift)
    got = first_result(f, (A, B, C))
    want = C.copy()
    name = f"{case.name}_srs_kc{kc}_shift{shift}"
    olog.run(name, oracle.igemm_srs, A, B, want, kc, shift, False)
    exact = bool(np.array_equal(got, want))
    del got, want
    m, n, k = case.m, case.n, case.k
    nblocks = 1 if (kc == 0 or kc >= k) else -(-k // kc)
    ops = 2.0 * m * n * k
    nbytes = A.nbytes + B.nbytes + 4.0 * m * n * nblocks
    memory_bound = roofline(ops, nbytes, 2, 1.0)[0] == "hbm"
    t, nsets, cycled = replay_sets(f, (A, B, C), A.nbytes + B.nbytes + C.nbytes, memory_bound,
                                   min_per_graph=10 if nblocks > 4 else 40)
    import torch
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    aligned = 1 << 12   # stands for a 16-byte aligned buffer; never dereferenced
    ws = ig.igemm_srs_query(2, m, n, k, aligned, k, aligned, n, aligned, n, kc, ncu)
    e = entry(t, ops, nbytes, 2, "packed" if ws > 0 else "fused", cycled, exact)
    details.append({"name": name, "m": m, "n": n, "k": k, "kc": kc, "blocks": nblocks,
                    "workspace_bytes": ws, "sets": nsets, **e})
    return name, e


def bench_conv(case, olog, details):
    """One convolution (implicit GEMM: IM2ROW gathered in the kernel); the
    roofline counts the lowered GEMM's multiply-adds and the unique bytes of
    X, W and Y (read and written)."""
    import numpy as np

    import oracle
    import paper_2302_07594_amd as ig
    import workloads
    X, W, Y = workloads.generate_conv(case)
    es = 2 if case.dtype == "i16" else 1
    kw = dict(stride=case.stride, pad=case.pad, dil=case.dil)
    f = lambda x, w, y: ig.conv2d(x, w, y, **kw)
    got = first_result(f, (X, W, Y))
    want = Y.copy()
    olog.run(case.name, oracle.conv2d, X, W, want, case.stride, case.pad, case.dil)
    exact = bool(np.array_equal(got, want))
    del got, want
    m, n, k = case.gemm_shape()
    ops = 2.0 * m * n * k
    nbytes = X.nbytes + W.nbytes + 2.0 * Y.nbytes
    memory_bound = roofline(ops, nbytes, es, 1.0)[0] == "hbm"
    t, nsets, cycled = replay_sets(f, (X, W, Y), X.nbytes + W.nbytes + Y.nbytes, memory_bound,
                                   min_per_graph=40 if case.n == 1 else 10)
    d = ig.conv_desc(case.n, case.h, case.w, case.c, case.k, case.r, case.s, case.stride,
                     case.pad, case.dil)
    plan = ig.igemm_conv2d_query_plan(es, d)
    e = entry(t, ops, nbytes, es, f"{plan['kernel_name']}/{plan['split']}", cycled, exact)
    details.append({"name": case.name, "gemm": [m, n, k], "plan": plan, "sets": nsets, **e})
    return e


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_one_thread_seconds():
    """The oracle on the int16 256^3 workload with one OpenMP thread, in a
    child process (the thread count is fixed when the runtime starts)."""
    code = ("import time, workloads, oracle\n"
            "A, B, C = workloads.generate(workloads.WORKLOADS['i16_256'].cases[0])\n"
            "t = time.perf_counter(); oracle.igemm(A, B, C)\n"
            "print(time.perf_counter() - t, oracle.num_threads())\n")
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    if r.returncode != 0:
        return None
    secs, threads = r.stdout.split()
    return round(float(secs), 4) if int(threads) == 1 else None


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-extra", action="store_true", help="skip the per-config table")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--details", default=None, help="write every per-config record here")
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
    log("bench: int16 4096^3 step")
    A, B, C0 = workloads.generate(case)
    Ad = torch.from_numpy(A).cuda()
    Bd = torch.from_numpy(B).cuda()
    Cd = torch.from_numpy(C0).cuda()
    # First launch on the pristine C; its result is compared with the oracle.
    ig.gemm_i16(Ad, Bd, Cd)
    torch.cuda.synchronize()
    C_first = Cd.cpu().numpy()
    plan = ig.igemm_query_plan(2, m, n, k, Ad, k, Bd, n, Cd, n)

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
    mf = measured_mfma("i16")

    out = {
        "metric": "int16 GEMM C+=A.B throughput on 1 MI355X (int8 MFMA limb split), TOPS",
        "value": round(value, 2), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int16", "data": "synthetic",
        "config": {
            "workload": "int16 GEMM C += A.B, m=n=k=4096, row-major, A,B uniform over the full "
                        "int16 range, C uniform in [-2^20,2^20], int32 wraparound, seed 1",
            "kernel": plan["kernel_name"], "workspace_bytes": plan["workspace_bytes"],
        },
        "roofline": {
            "bound": "mfma", "achieved": round(ach, 1), "peak": PEAK_I16_TOPS, "unit": "TOPS",
            "frac": round(ach / PEAK_I16_TOPS, 4), "traffic": measured_traffic("i16"),
            "kernel": "igemm_packed<int16,128x128> multiply, on packed operands",
            "peak_basis": "5000 TOPS int8 MFMA / 4 limb products",
            "kernel_us": round(mult * 1e6, 2), "pack_us": round(pack_t * 1e6, 2),
            "step_device_us": round(step_dev * 1e6, 2),
            "step_frac": round(value / PEAK_I16_TOPS, 4),
            **({"mfma_busy": mf["mfma_busy"], "clk_ghz": mf["clock_ghz"]} if mf else {}),
        },
    }
    olog = OracleLog()
    if not args.no_cpu_baseline:
        import oracle
        log("bench: CPU oracle on the whole int16 4096^3 workload")
        want = C0.copy()
        olog.run(case.name, oracle.igemm, A, B, want)
        secs = olog.seconds[case.name]
        out["cpu_baseline"] = {
            "value": round(ops / secs / 1e12, 6), "unit": "TOPS",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"the whole {m}x{n}x{k} int16 workload ({m * n * k:.3g} multiply-adds, "
                      f"{secs:.2f} s)",
            "exact": bool(np.array_equal(C_first, want)),
            "cpu_model": cpu_model(),
            "i16_256_1thread_s": oracle_one_thread_seconds(),
        }
        del want
    del Ad, Bd, Cd, C_first
    torch.cuda.empty_cache()
    details = []
    if not args.no_extra:
        import oracle  # noqa: F401  (per-config results are checked against it)
        per = {}
        for wname in ("i16_256", "i8_8192", "i16_conv", "i8_skinny", "i16_skinny",
                      "i16_paper"):
            for c in workloads.WORKLOADS[wname].cases:
                log(f"bench: {c.name}")
                per[c.name] = bench_gemm(c, olog, details)
        for c, kc in ((workloads.WORKLOADS["i16_paper"].cases[0], 290),
                      (workloads.WORKLOADS["i16_4096"].cases[0], 256)):
            log(f"bench: {c.name} int16 output, kc {kc}")
            name, e = bench_srs(c, kc, 0, olog, details)
            per[name] = e
        for c in workloads.CONV2D_CASES + workloads.CONV2D_B32_CASES:
            log(f"bench: {c.name}")
            per[c.name] = bench_conv(c, olog, details)
        cbw = copy_bandwidth()
        out["copy_GBs"] = round(cbw / 1e9, 1)
        for e in per.values():
            if e["bound"] == "hbm":
                e["fc"] = round(e["GBs"] * 1e9 / cbw, 4)
        if "cpu_baseline" in out:
            out["cpu_baseline"]["per_config_s"] = olog.seconds
        out["all_exact"] = all(e["exact"] for e in per.values()) and \
            out.get("cpu_baseline", {}).get("exact", True)
        out["per_config"] = per
    if args.details:
        with open(args.details, "w") as f:
            json.dump({"headline": out, "per_config": details}, f, indent=1, default=str)
    print(json.dumps(out, separators=(",", ":")), flush=True)


if __name__ == "__main__":
    main()
