"""Helpers for GPU parity tests: run the HIP path through the C ABI on
device copies of numpy operands and return the host result."""
from __future__ import annotations

import numpy as np

NP_TO_ES = {np.dtype(np.int16): 2, np.dtype(np.int8): 1}


def to_device(x: np.ndarray, offset_elems: int = 0):
    """Device copy of a 2-D array; with offset_elems > 0 the copy starts that
    many elements into a larger allocation (a misaligned base address)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    if offset_elems == 0:
        return t.cuda()
    flat = torch.empty(x.size + offset_elems, dtype=t.dtype, device="cuda")
    flat[:offset_elems] = 0
    view = flat[offset_elems:].view(x.shape)
    view.copy_(t.cuda())
    return view


def gpu_gemm(A, B, C, m, n, k, kernel=-1, split=-1, offsets=(0, 0, 0), stream=None,
             check_status=True, workspace="auto"):
    """Run C += A.B on the GPU. A, B, C are full numpy arrays whose row length
    is the leading dimension; the logical shapes are m x k, k x n, m x n.
    workspace="auto" passes a workspace of the planned size to the _ws entry
    point when the plan (with this kernel and split) packs the operands, and
    calls the _ex entry point otherwise; workspace=None calls the _ex entry
    point (no workspace); a device tensor is passed to the _ws entry point.
    Returns (status, C after the call as numpy)."""
    import torch

    import paper_2302_07594_amd as ig
    es = NP_TO_ES[A.dtype]
    Ad = to_device(A, offsets[0])
    Bd = to_device(B, offsets[1])
    Cd = to_device(C, offsets[2])
    lda, ldb, ldc = A.shape[1], B.shape[1], C.shape[1]
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    if isinstance(workspace, str) and workspace == "auto":
        workspace = None
        if m and n and k:
            plan = ig.igemm_query_plan(es, m, n, k, Ad, lda, Bd, ldb, Cd, ldc,
                                       torch.cuda.get_device_properties(0).multi_processor_count,
                                       kernel, split)
            if plan["workspace_bytes"] > 0:
                workspace = torch.empty(plan["workspace_bytes"], dtype=torch.uint8,
                                        device="cuda")
    if workspace is None:
        fn = ig.igemm_i16_ex if es == 2 else ig.igemm_i8_ex
        st = fn(m, n, k, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, Cd.data_ptr(), ldc, s,
                kernel, split)
    else:
        fn = ig.igemm_i16_ws if es == 2 else ig.igemm_i8_ws
        st = fn(m, n, k, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, Cd.data_ptr(), ldc, s,
                kernel, split, workspace.data_ptr(), workspace.numel())
    torch.cuda.synchronize()
    if check_status and st != 0:
        raise AssertionError(f"status {st}: {ig.igemm_strerror(st)}")
    return st, Cd.cpu().numpy()


def oracle_gemm(A, B, C, m, n, k):
    """Oracle result on the same padded arrays (padding untouched)."""
    import oracle
    out = C.copy()
    oracle.igemm(A[:m, :k], B[:k, :n], out[:m, :n])
    return out


def describe_mismatch(got, want, limit=5):
    bad = np.argwhere(got != want)
    lines = [f"{len(bad)} mismatching elements"]
    for (i, j) in bad[:limit]:
        lines.append(f"  [{i},{j}] got {got[i, j]} want {want[i, j]}")
    return "\n".join(lines)


def general_kernels(es):
    """Kernel indices of the operand type that take any shape and alignment
    (all but the direct and small-output kernels, whose preconditions have
    tests of their own)."""
    import paper_2302_07594_amd as ig
    return [k for k in ig.kernels_for(es) if not restricted(ig.igemm_kernel_name(k))]


def restricted(name):
    """Kernels that take only aligned operands and whole k-tiles."""
    return "direct" in name or "small" in name or "i16_stream" in name
