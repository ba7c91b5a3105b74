"""igemm_i16_noalloc (the packed path on the library's static device scratch
array, for callers that cannot allocate) against igemm_i16_ws with a caller
workspace, bit for bit, through the C ABI: two calls in a row, the second
with a smaller product, so the second finds the first's contents in the
array; then a product too large for the array, refused untouched."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, oracle_gemm

pytestmark = pytest.mark.gpu


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _run_both(m, n, k, seed):
    """(noalloc result, _ws result, host operands) for one product; both
    calls start from the same C."""
    import torch
    ig = _ig()
    A, B, C = workloads.random_operands("i16", m, n, k, seed=seed)
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    C1, C2 = torch.from_numpy(C).cuda(), torch.from_numpy(C).cuda()
    s = torch.cuda.current_stream().cuda_stream
    plan = ig.igemm_query_plan(2, m, n, k, Ad, k, Bd, n, C1, n,
                               torch.cuda.get_device_properties(0).multi_processor_count)
    assert plan["packed"] == 1 and 0 < plan["workspace_bytes"] <= ig.IGEMM_NOALLOC_SCRATCH_BYTES
    st = ig.igemm_i16_noalloc(m, n, k, Ad, k, Bd, n, C1, n, s)
    assert st == ig.IGEMM_OK, ig.igemm_strerror(st)
    ws = torch.empty(plan["workspace_bytes"], dtype=torch.uint8, device="cuda")
    st = ig.igemm_i16_ws(m, n, k, Ad, k, Bd, n, C2, n, s, -1, -1, ws, ws.numel())
    assert st == ig.IGEMM_OK, ig.igemm_strerror(st)
    torch.cuda.synchronize()
    return C1.cpu().numpy(), C2.cpu().numpy(), (A, B, C)


def test_noalloc_matches_ws_twice_then_refuses_oversize():
    import torch
    ig = _ig()
    # 1: the largest product the array holds (int16 4096^3, 64.1 MiB packed)
    got, ref, _ = _run_both(4096, 4096, 4096, seed=3001)
    assert np.array_equal(got, ref), describe_mismatch(got, ref)
    # 2: a smaller product on the array the first call left behind
    got, ref, (A, B, C) = _run_both(2048, 2560, 1000, seed=3002)
    assert np.array_equal(got, ref), describe_mismatch(got, ref)
    want = oracle_gemm(A, B, C, 2048, 2560, 1000)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    # 3: a product whose packed operands exceed the array: refused, C untouched
    m, n, k = 4096, 8192, 4096
    Ad = torch.zeros((m, k), dtype=torch.int16, device="cuda")
    Bd = torch.zeros((k, n), dtype=torch.int16, device="cuda")
    Cd = torch.full((m, n), 7, dtype=torch.int32, device="cuda")
    st = ig.igemm_i16_noalloc(m, n, k, Ad, k, Bd, n, Cd, n)
    assert st == ig.IGEMM_ESCRATCH
    torch.cuda.synchronize()
    assert bool((Cd == 7).all())
    # ... and runs with an explicit fused kernel, which needs no scratch
    kid = [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == "i16_128x128"][0]
    assert ig.igemm_i16_noalloc(m, n, k, Ad, k, Bd, n, Cd, n, None, kid, -1) == ig.IGEMM_OK
    torch.cuda.synchronize()
    assert bool((Cd == 7).all())
