"""The library's launches inside a captured HIP graph: every replay must
match the eager result (the calls enqueue kernels only -- no memset nodes)."""
import numpy as np
import pytest

import workloads
from gpu_util import oracle_gemm

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt,shape,split", [("i16", (130, 260, 300), -1), ("i8", (40, 300, 700), 5),
                                            ("i16", (256, 256, 256), 1),
                                            ("i16", (1100, 1030, 1200), -1),
                                            ("i8", (1030, 1100, 1300), -1),
                                            ("i8", (32, 11008, 4096), -1),
                                            ("i16", (8, 4096, 4096), -1)])
def test_graph_replays_match_eager(dt, shape, split):
    """(1100, 1030, 1200) and (1030, 1100, 1300) take the packed path; its
    workspace comes from torch's caching allocator, which is capture-aware.
    (32, 11008, 4096) int8 takes the streaming kernel's ring variant (two
    slices of 32 k-steps), (8, 4096, 4096) int16 the int16 streaming
    kernel."""
    import torch
    import paper_2302_07594_amd as ig
    m, n, k = shape
    A, B, C0 = workloads.random_operands(dt, m, n, k, seed=31)
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    Cd = torch.from_numpy(C0).cuda()
    f = ig.gemm_i16 if dt == "i16" else ig.gemm_i8
    f(Ad, Bd, Cd, split=split)              # warm up outside the graph
    torch.cuda.synchronize()
    Cd.copy_(torch.from_numpy(C0).cuda())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        f(Ad, Bd, Cd, split=split)
    torch.cuda.synchronize()
    # the capture did not run the kernel
    assert np.array_equal(Cd.cpu().numpy(), C0)
    expect = C0.copy()
    for rep in range(4):
        g.replay()
        torch.cuda.synchronize()
        expect = oracle_gemm(A, B, expect, m, n, k)
        assert np.array_equal(Cd.cpu().numpy(), expect), f"replay {rep}"
        # eager work between replays
        f(Ad, Bd, Cd, split=split)
        torch.cuda.synchronize()
        expect = oracle_gemm(A, B, expect, m, n, k)
        assert np.array_equal(Cd.cpu().numpy(), expect), f"eager after replay {rep}"
