"""Profiling driver: run one workload (or a plain copy) a few times so that
``rocprofv3`` can trace it, and summarize the resulting CSV files.

Usage (the program itself goes after ``rocprofv3 ... --``):
    python paper_2302_07594_amd/profile_run.py gemm <workload> [iters] [case]
    python paper_2302_07594_amd/profile_run.py conv <layer> [iters]
    python paper_2302_07594_amd/profile_run.py copy <MiB> [iters]
    python paper_2302_07594_amd/profile_run.py summarize <rocprof output dir>

``gemm`` runs the library's igemm call on the named workload's case (inputs
generated as in the benchmark, C reset is not needed for timing); ``conv``
runs the convolution entry point on one of the six network layers (index
into ``workloads.CONV2D_CASES``).
``copy`` runs a device-to-device copy of a tensor of the given size; its
FETCH_SIZE / WRITE_SIZE readings calibrate the counters against a known byte
count. ``summarize`` prints per-kernel average durations from a
``*_kernel_stats.csv`` and per-dispatch counter values from a
``*_counter_collection.csv`` found under the directory.
"""
from __future__ import annotations

import csv
import glob
import os
import sys
from collections import defaultdict

# Runnable as a file from any directory (rocprofv3 is started from /tmp).
_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if _ROOT not in sys.path:
    sys.path.insert(0, _ROOT)


def _gemm(wname: str, iters: int, case_idx: int) -> None:
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    case = workloads.WORKLOADS[wname].cases[case_idx]
    A, B, C = workloads.generate(case)
    Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
    f = ig.gemm_i16 if case.dtype == "i16" else ig.gemm_i8
    for _ in range(iters):
        f(Ad, Bd, Cd)
    torch.cuda.synchronize()
    print(f"ran {case.name} x{iters}", flush=True)


def _conv(layer: int, iters: int) -> None:
    import torch

    import paper_2302_07594_amd as ig
    import workloads
    case = workloads.CONV2D_CASES[layer]
    X, W, Y = workloads.generate_conv(case)
    Xd, Wd, Yd = (torch.from_numpy(x).cuda() for x in (X, W, Y))
    for _ in range(iters):
        ig.conv2d(Xd, Wd, Yd, stride=case.stride, pad=case.pad, dil=case.dil)
    torch.cuda.synchronize()
    print(f"ran {case.name} x{iters}", flush=True)


def _copy(mib: int, iters: int) -> None:
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(iters):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x{iters}", flush=True)


def _summarize(d: str) -> None:
    for f in sorted(glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)):
        print(f"# kernel stats: {os.path.relpath(f, d)}")
        for r in csv.DictReader(open(f)):
            print(f"{r['Name'][:110]} | calls {r['Calls']} | avg {float(r['AverageNs']) / 1e3:.2f} us"
                  f" | min {float(r['MinNs']) / 1e3:.2f} us | max {float(r['MaxNs']) / 1e3:.2f} us")
    for f in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
        print(f"# counters: {os.path.relpath(f, d)}")
        per = defaultdict(lambda: defaultdict(float))
        names = {}
        for r in csv.DictReader(open(f)):
            key = int(r["Dispatch_Id"])
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            names[key] = r["Kernel_Name"]
        for key in sorted(per):
            vals = ", ".join(f"{c}={v:.1f}" for c, v in sorted(per[key].items()))
            print(f"dispatch {key} | {names[key][:90]} | {vals}")


def main(argv) -> None:
    if len(argv) < 2:
        print(__doc__)
        sys.exit(2)
    cmd = argv[1]
    if cmd == "gemm":
        _gemm(argv[2], int(argv[3]) if len(argv) > 3 else 3, int(argv[4]) if len(argv) > 4 else 0)
    elif cmd == "conv":
        _conv(int(argv[2]), int(argv[3]) if len(argv) > 3 else 3)
    elif cmd == "copy":
        _copy(int(argv[2]), int(argv[3]) if len(argv) > 3 else 3)
    elif cmd == "summarize":
        _summarize(argv[2])
    else:
        print(__doc__)
        sys.exit(2)


if __name__ == "__main__":
    main(sys.argv)
