"""GPU parity of the pack-B-once path (the fixed operand packed once, then
multiplied with many A of any row count) against the CPU oracle, bit-exact,
through the C ABI and the tensor wrappers."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, oracle_gemm, to_device

pytestmark = pytest.mark.gpu

PACKED = {"i16": "i16_packed_128x128", "i8": "i8_packed_256x256"}
ES = {"i16": 2, "i8": 1}


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _kid(dt):
    ig = _ig()
    return [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == PACKED[dt]][0]


def _aligned(nbytes):
    import torch
    t = torch.empty(nbytes + 256, dtype=torch.uint8, device="cuda")
    off = (-t.data_ptr()) % 256
    return t[off:off + nbytes]


def _pack_b_abi(dt, B, n, k):
    """Pack B through the C ABI into a caller buffer; returns (buffer, bytes)."""
    ig = _ig()
    es, kid = ES[dt], _kid(dt)
    nbytes = ig.igemm_query_plan(es, 1, n, k, None, k, None, B.shape[1], None, n,
                                 kernel=kid)["packed_b_bytes"]
    Bd = to_device(B)
    buf = _aligned(nbytes)
    fn = ig.igemm_pack_b_i16 if es == 2 else ig.igemm_pack_b_i8
    st = fn(n, k, Bd, B.shape[1], kid, buf, nbytes, None)
    assert st == 0, ig.igemm_strerror(st)
    return buf, nbytes


def _mul_abi(dt, A, m, n, k, buf, nbytes, C, with_ws=True, a_offset=0):
    """igemm_*_packed_b through the C ABI. with_ws=False passes no workspace
    (valid only when A needs no packed copy); returns (status, C)."""
    import torch
    ig = _ig()
    es, kid = ES[dt], _kid(dt)
    Ad = to_device(A, a_offset)
    Cd = to_device(C)
    lda, ldc = A.shape[1], C.shape[1]
    ws, ws_bytes = None, 0
    if with_ws:
        ws_bytes = ig.igemm_query_plan(es, m, n, k, Ad, lda, None, n, Cd, ldc,
                                       kernel=kid)["packed_a_bytes"]
        ws = _aligned(max(ws_bytes, 1)) if ws_bytes > 0 else None
    fn = ig.igemm_i16_packed_b if es == 2 else ig.igemm_i8_packed_b
    st = fn(m, n, k, Ad, lda, buf, nbytes, Cd, ldc, kid, ws, ws_bytes, None)
    torch.cuda.synchronize()
    return st, Cd.cpu().numpy()


def _mul_ok(*args, **kw):
    st, got = _mul_abi(*args, **kw)
    assert st == 0, _ig().igemm_strerror(st)
    return got


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_b_without_workspace(dt):
    """No workspace: refused (C untouched) when A needs a packed copy; int8 A
    that the multiply reads in place (aligned, 256-row multiple, k a multiple
    of 256) needs none and runs."""
    ig = _ig()
    n, k = 520, 768
    B = workloads.random_operands(dt, 1, n, k, seed=1211)[1]
    buf, nbytes = _pack_b_abi(dt, B, n, k)
    A, _, C = workloads.random_operands(dt, 300, n, k, seed=1212)
    st, got = _mul_abi(dt, A, 300, n, k, buf, nbytes, C, with_ws=False)
    assert st == ig.IGEMM_EINVAL and np.array_equal(got, C)
    if dt == "i8":
        A, _, C = workloads.random_operands(dt, 512, n, k, seed=1213)
        st, got = _mul_abi(dt, A, 512, n, k, buf, nbytes, C, with_ws=False)
        want = oracle_gemm(A, B, C, 512, n, k)
        assert st == 0 and np.array_equal(got, want), describe_mismatch(got, want)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_pack_b_once_many_a(dt):
    """One packed B, then A of 1, 129, 300 and 512 rows (int8 512 rows and
    k = 768 reads A in place) and padded leading dimensions: every product
    matches the oracle."""
    n, k = 520, 768
    B = workloads.random_operands(dt, 1, n, k, seed=1201, ldb=n + 5)[1]
    buf, nbytes = _pack_b_abi(dt, B, n, k)
    for i, m in enumerate((1, 129, 300, 512)):
        lda = k + (0 if m == 512 else 3)
        A, _, C = workloads.random_operands(dt, m, n, k, seed=1300 + i, lda=lda, ldc=n + 2)
        got = _mul_ok(dt, A, m, n, k, buf, nbytes, C)
        want = oracle_gemm(A, B, C, m, n, k)
        assert np.array_equal(got, want), f"m={m}\n" + describe_mismatch(got, want)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_b_misaligned_a(dt):
    n, k = 300, 1000
    B = workloads.random_operands(dt, 1, n, k, seed=1401)[1]
    buf, nbytes = _pack_b_abi(dt, B, n, k)
    A, _, C = workloads.random_operands(dt, 200, n, k, seed=1402)
    got = _mul_ok(dt, A, 200, n, k, buf, nbytes, C, a_offset=1)
    want = oracle_gemm(A, B, C, 200, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


@pytest.mark.parametrize("value", [-32768, 32767])
def test_packed_b_int16_extremes_two_chunks(value):
    """All-extreme int16 operands with k = 33000 (two multiply launches): the
    corrections packed with B serve the whole k range."""
    m, n, k = 130, 140, 33000
    A = np.full((m, k), value, dtype=np.int16)
    B = np.full((k, n), value, dtype=np.int16)
    C = np.zeros((m, n), dtype=np.int32)
    buf, nbytes = _pack_b_abi("i16", B, n, k)
    got = _mul_ok("i16", A, m, n, k, buf, nbytes, C)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_b_buffer_is_read_only(dt):
    """Multiplies only read the packed B: its bytes are unchanged after
    several calls, and a second identical call gives the same result."""
    import torch
    n, k = 384, 700
    B = workloads.random_operands(dt, 1, n, k, seed=1501)[1]
    buf, nbytes = _pack_b_abi(dt, B, n, k)
    torch.cuda.synchronize()
    before = buf.clone()
    A, _, C = workloads.random_operands(dt, 257, n, k, seed=1502)
    r1 = _mul_ok(dt, A, 257, n, k, buf, nbytes, C)
    r2 = _mul_ok(dt, A, 257, n, k, buf, nbytes, C)
    assert torch.equal(buf, before)
    assert np.array_equal(r1, r2)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_b_equals_one_shot_call(dt):
    """The tensor wrappers: pack_b + gemm_packed_b gives bit for bit what
    the one-call packed path gives."""
    import torch
    ig = _ig()
    m, n, k = 640, 700, 900
    A, B, C = workloads.random_operands(dt, m, n, k, seed=1601)
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    C1, C2 = torch.from_numpy(C).cuda(), torch.from_numpy(C).cuda()
    f = ig.gemm_i16 if dt == "i16" else ig.gemm_i8
    f(Ad, Bd, C1, kernel=_kid(dt))
    PB = ig.pack_b(Bd)
    del Bd
    ig.gemm_packed_b(Ad, PB, C2)
    torch.cuda.synchronize()
    assert torch.equal(C1, C2)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(C2.cpu().numpy(), want)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_b_in_graph(dt):
    """gemm_packed_b captured into a graph (A's packed copy from torch's
    allocator): every replay matches the oracle, with eager calls between."""
    import torch
    ig = _ig()
    m, n, k = 300, 520, 1000
    A, B, C0 = workloads.random_operands(dt, m, n, k, seed=1701)
    Ad, Cd = torch.from_numpy(A).cuda(), torch.from_numpy(C0).cuda()
    PB = ig.pack_b(torch.from_numpy(B).cuda())
    ig.gemm_packed_b(Ad, PB, Cd)          # warm up outside the graph
    torch.cuda.synchronize()
    Cd.copy_(torch.from_numpy(C0).cuda())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ig.gemm_packed_b(Ad, PB, Cd)
    torch.cuda.synchronize()
    assert np.array_equal(Cd.cpu().numpy(), C0)
    expect = C0.copy()
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        expect = oracle_gemm(A, B, expect, m, n, k)
        assert np.array_equal(Cd.cpu().numpy(), expect), f"replay {rep}"
        ig.gemm_packed_b(Ad, PB, Cd)
        torch.cuda.synchronize()
        expect = oracle_gemm(A, B, expect, m, n, k)
        assert np.array_equal(Cd.cpu().numpy(), expect), f"eager after replay {rep}"


def test_packed_b_wrapper_rejects_mismatch():
    import torch
    ig = _ig()
    PB = ig.pack_b(torch.zeros((64, 32), dtype=torch.int16, device="cuda"))
    with pytest.raises(ValueError):
        ig.gemm_packed_b(torch.zeros((8, 63), dtype=torch.int16, device="cuda"), PB,
                         torch.zeros((8, 32), dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        ig.gemm_packed_b(torch.zeros((8, 64), dtype=torch.int8, device="cuda"), PB,
                         torch.zeros((8, 32), dtype=torch.int32, device="cuda"))
