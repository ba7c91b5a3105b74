"""Parameter sweeps on MI355X that mirror the paper's experiments.

* k sweep -- the analogue of the paper's k_c sweep (Sec. 6.3, Fig. "kc_sweep"):
  there the micro-kernel's efficiency grows with k_c because the load and
  store of the C micro-tile are amortised over k_c rank-1 updates. Here the
  per-workgroup k range plays k_c: int16 m = n = k = 4096 on the fused
  128x128 kernel with s k slices gives each workgroup a k range of 4096/s and
  s read-add-writes (atomic adds) of its C tile; the packed kernel runs the
  whole k range at once.
* packed k sweep -- the same question for the kernels the automatic plan
  uses for large products: int16 m = n = 4096 with k = 256 ... 8192 on the
  packed path (pack + multiply per call) and on the direct kernel; here the
  whole k range of a call is one workgroup's range.
* kc sweep -- the int16-output update's block size (Sec. 5.2: the
  accumulator is converted to int16 at the end of every k_c block): int16
  4096^3 with k_c = 256 ... 4096, one packed launch converting at each block
  boundary.
* m sweep -- the analogue of the m_c sweep on the paper's GEMM
  (m, n, k) = (4096, 4096, 290) with n_c = n and k_c = k (Sec. 6.4, Fig.
  "mc_sweep"): there m_c is the height of the A block kept close to the
  tile; here it is the workgroup tile height (16, 32, 64, 128 rows).

Every point is timed by HIP-graph replay of one-call igemm_i16 launches over
rotating buffer sets (larger than the 256 MB last-level cache together), and
reported as TOPS (2mnk / time) and as a fraction of the int16 peak (the int8
matrix-core peak of 5000 TOPS divided by four limb products).

Usage: python -m paper_2302_07594_amd.sweep [k|kp|kc|m|all]
Prints one JSON object per point and a markdown table per sweep.
"""
from __future__ import annotations

import json
import os
import sys

_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if _ROOT not in sys.path:
    sys.path.insert(0, _ROOT)

PEAK_I16_TOPS = 5000.0 / 4
MALL_BYTES = 256 << 20


def _kid(ig, name):
    return [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == name][0]


def time_gemm(case, kernel=-1, split=-1, per_graph=20, reps=5):
    """Seconds per one-call launch of `case` (a workloads.Case) with the given
    kernel and k-slice count, by graph replay over rotating buffer sets."""
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    A, B, C = workloads.generate(case)
    set_bytes = A.nbytes + B.nbytes + C.nbytes
    nsets = max(1, min(16, -(-2 * MALL_BYTES // set_bytes)))
    base = [torch.from_numpy(x).cuda() for x in (A, B, C)]
    sets = [base] + [[t.clone() for t in base] for _ in range(nsets - 1)]
    f = ig.gemm_i16 if case.dtype == "i16" else ig.gemm_i8
    for i in range(2):
        f(*sets[i % nsets], kernel=kernel, split=split)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            f(*sets[i % nsets], kernel=kernel, split=split)
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / (reps * per_graph)
    plan = ig.igemm_query_plan(2 if case.dtype == "i16" else 1, case.m, case.n, case.k,
                               kernel=kernel, split=split)
    del sets, base, g
    torch.cuda.empty_cache()
    return t, plan


def _point(sweep, label, case, kernel=-1, split=-1):
    t, plan = time_gemm(case, kernel, split)
    tops = 2.0 * case.m * case.n * case.k / t / 1e12
    rec = {"sweep": sweep, "point": label, "m": case.m, "n": case.n, "k": case.k,
           "kernel": plan["kernel_name"], "split": plan["split"],
           "k_range_per_workgroup": plan["k_chunk"], "us": round(t * 1e6, 2),
           "TOPS": round(tops, 1), "frac_of_int16_peak": round(tops / PEAK_I16_TOPS, 4)}
    print(json.dumps(rec), flush=True)
    return rec


def k_sweep():
    import paper_2302_07594_amd as ig
    import workloads
    case = workloads.WORKLOADS["i16_4096"].cases[0]
    fused = _kid(ig, "i16_128x128")
    out = []
    for s in (64, 32, 16, 8, 4, 2, 1):
        out.append(_point("k", f"fused 128x128, {s} k slices", case, fused, s))
    out.append(_point("k", "packed 128x128", case, _kid(ig, "i16_packed_128x128")))
    return out


def _case_4096(k):
    import workloads
    base = workloads.WORKLOADS["i16_4096"].cases[0]
    return workloads.Case(f"i16_4096x4096x{k}", "i16", 4096, 4096, k, base.a, base.b, base.c,
                          base.seed)


def packed_k_sweep():
    import paper_2302_07594_amd as ig
    out = []
    for k in (256, 512, 1024, 2048, 4096, 8192):
        case = _case_4096(k)
        out.append(_point("kp", f"packed, k = {k}", case, _kid(ig, "i16_packed_128x128")))
        out.append(_point("kp", f"direct, k = {k}", case, _kid(ig, "i16_direct_128x128")))
    return out


def time_srs(case, kc, per_graph=10, reps=5):
    """Seconds per one-call int16-output update (gemm_srs, shift 0) of `case`
    with block size kc, by graph replay over rotating buffer sets."""
    import numpy as np
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    A, B, _ = workloads.generate(case)
    C = np.zeros((case.m, case.n), dtype=np.int16)
    set_bytes = A.nbytes + B.nbytes + C.nbytes
    nsets = max(1, min(16, -(-2 * MALL_BYTES // set_bytes)))
    base = [torch.from_numpy(x).cuda() for x in (A, B, C)]
    sets = [base] + [[t.clone() for t in base] for _ in range(nsets - 1)]
    for i in range(2):
        ig.gemm_srs(*sets[i % nsets], kc=kc)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(per_graph):
            ig.gemm_srs(*sets[i % nsets], kc=kc)
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / (reps * per_graph)
    del sets, base, g
    torch.cuda.empty_cache()
    return t


def kc_sweep():
    import workloads
    case = workloads.WORKLOADS["i16_4096"].cases[0]
    out = []
    for kc in (256, 512, 1024, 2048, 4096):
        t = time_srs(case, kc)
        tops = 2.0 * case.m * case.n * case.k / t / 1e12
        rec = {"sweep": "kc", "point": f"k_c = {kc}", "m": case.m, "n": case.n, "k": case.k,
               "kernel": "i16_packed_128x128 (int16 output)", "split": 1,
               "k_range_per_workgroup": case.k, "us": round(t * 1e6, 2), "TOPS": round(tops, 1),
               "frac_of_int16_peak": round(tops / PEAK_I16_TOPS, 4)}
        print(json.dumps(rec), flush=True)
        out.append(rec)
    return out


def m_sweep():
    import paper_2302_07594_amd as ig
    import workloads
    case = workloads.WORKLOADS["i16_paper"].cases[0]
    out = []
    for name in ("i16_16x128", "i16_32x128", "i16_64x64", "i16_128x128"):
        out.append(_point("m", f"{name}, whole k", case, _kid(ig, name), 1))
    out.append(_point("m", "automatic plan", case))
    return out


def table(rows):
    lines = ["| point | kernel | k slices | k per workgroup | time | TOPS | of int16 peak |",
             "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['point']} | `{r['kernel']}` | {r['split']} | "
                     f"{r['k_range_per_workgroup']} | {r['us']:.1f} us | {r['TOPS']:.1f} | "
                     f"{r['frac_of_int16_peak']:.3f} |")
    return "\n".join(lines)


def main(argv):
    which = argv[1] if len(argv) > 1 else "all"
    if which in ("k", "all"):
        print(table(k_sweep()), flush=True)
    if which in ("kp", "all"):
        print(table(packed_k_sweep()), flush=True)
    if which in ("kc", "all"):
        print(table(kc_sweep()), flush=True)
    if which in ("m", "all"):
        print(table(m_sweep()), flush=True)


if __name__ == "__main__":
    main(sys.argv)
