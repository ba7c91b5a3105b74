"""GPU parity of the pack-then-multiply path (pack kernels into a workspace,
then the DMA-fed matrix-core kernel) against the CPU oracle, bit-exact, and
its workspace handling: caller workspaces (the library allocates none),
too-small and misaligned workspaces, refusal of the packed kernels without a
workspace, graph capture."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, gpu_gemm, oracle_gemm

pytestmark = pytest.mark.gpu

PACKED = {"i16": "i16_packed_128x128", "i8": "i8_packed_256x256"}


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _kid(dt):
    ig = _ig()
    return [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == PACKED[dt]][0]


def _workspace(nbytes):
    import torch
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")


def _check(dt, A, B, C, m, n, k, **kw):
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(dt), **kw)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    return got


SHAPES = [
    (1, 1, 1),
    (7, 300, 5),              # k far below one 256-element pack unit
    (129, 257, 255),          # one more than a tile in m and n, k just below 256
    (256, 256, 256),          # exactly one int8 tile
    (300, 520, 1000),         # several tiles, ragged everywhere
    (640, 384, 2304),         # tile multiples (int8 A taken unpacked when aligned)
]


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("shape", SHAPES, ids=["x".join(map(str, s)) for s in SHAPES])
def test_packed_ragged(dt, shape):
    m, n, k = shape
    A, B, C = workloads.random_operands(dt, m, n, k, seed=600 + m + 3 * n + 7 * k)
    _check(dt, A, B, C, m, n, k)


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("shape", SHAPES[2:5], ids=["x".join(map(str, s)) for s in SHAPES[2:5]])
def test_packed_caller_workspace(dt, shape):
    ig = _ig()
    m, n, k = shape
    A, B, C = workloads.random_operands(dt, m, n, k, seed=700 + m + n + k)
    es = 2 if dt == "i16" else 1
    need = ig.igemm_query_plan(es, m, n, k, kernel=_kid(dt))["workspace_bytes"]
    ws = _workspace(need)
    ws.fill_(0x5A)   # stale contents must not matter
    _check(dt, A, B, C, m, n, k, workspace=ws)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_small_or_misaligned_workspace_rejected(dt):
    ig = _ig()
    m, n, k = 200, 300, 500
    A, B, C = workloads.random_operands(dt, m, n, k, seed=41)
    es = 2 if dt == "i16" else 1
    need = ig.igemm_query_plan(es, m, n, k, kernel=_kid(dt))["workspace_bytes"]
    ws = _workspace(need + 512)
    st, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(dt), workspace=ws[: need - 256],
                       check_status=False)
    assert st == ig.IGEMM_ENOMEM and np.array_equal(got, C)
    st, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(dt), workspace=ws[16:],
                       check_status=False)
    assert st == ig.IGEMM_EINVAL and np.array_equal(got, C)


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("offsets", [(1, 0, 0), (0, 1, 0), (1, 1, 1)])
def test_packed_misaligned_operands(dt, offsets):
    m, n, k = 260, 270, 600
    A, B, C = workloads.random_operands(dt, m, n, k, seed=43, lda=k + 3, ldb=n + 1, ldc=n + 2)
    got = _check(dt, A, B, C, m, n, k, offsets=offsets)
    assert np.array_equal(got[:, n:], C[:, n:])


@pytest.mark.parametrize("value", [-32768, 32767])
def test_packed_int16_extremes_multi_chunk(value):
    """k = 40000 > 32768: two main-kernel launches over one packing; every
    limb sum is at its bound."""
    m, n, k = 40, 70, 40000
    A = np.full((m, k), value, np.int16)
    B = np.full((k, n), value, np.int16)
    C = np.zeros((m, n), np.int32)
    got = _check("i16", A, B, C, m, n, k)
    assert np.all(got == got[0, 0])


@pytest.mark.parametrize("value", [-128, 127])
def test_packed_int8_extremes_multi_chunk(value):
    m, n, k = 33, 65, 70000
    A = np.full((m, k), value, np.int8)
    B = np.full((k, n), value, np.int8)
    C = np.full((m, n), 2 ** 31 - 1000, np.int32)
    _check("i8", A, B, C, m, n, k)


# k counts whose k-tiles of 64 are not a multiple of four. int16 with k up to
# 512 skips the MFMAs of the zero tiles (eight-wave kernel: k = 1, 130, 290,
# 330, 420); beyond it, it multiplies only the tiles that hold data when the
# padding spans three of them (1300: 21 tiles, through the tail chosen at run
# time) and the zero padding up to a multiple of four otherwise (1345).
RAGGED_K = [1, 130, 290, 330, 420, 1300, 1345]


@pytest.mark.parametrize("k", RAGGED_K)
def test_packed_int16_ragged_k_tiles(k):
    m, n = 200, 300
    A, B, C = workloads.random_operands("i16", m, n, k, seed=800 + k)
    _check("i16", A, B, C, m, n, k)


@pytest.mark.parametrize("value", [-32768, 32767])
def test_packed_int16_ragged_k_tiles_extremes(value):
    """Every limb sum at its bound with a ragged tile count (k = 290)."""
    m, n, k = 140, 130, 290
    A = np.full((m, k), value, np.int16)
    B = np.full((k, n), value, np.int16)
    C = np.zeros((m, n), np.int32)
    got = _check("i16", A, B, C, m, n, k)
    assert np.all(got == got[0, 0])


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_random_multi_chunk(dt):
    m, n, k = 130, 200, 33000
    A, B, C = workloads.random_operands(dt, m, n, k, seed=47)
    _check(dt, A, B, C, m, n, k)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_packed_matches_fused(dt):
    """Same inputs through the packed kernel and every other kernel of the
    type (k a multiple of 256, so that the direct kernel takes it too)."""
    ig = _ig()
    m, n, k = 300, 400, 1536
    A, B, C = workloads.random_operands(dt, m, n, k, seed=49)
    _, ref = gpu_gemm(A, B, C, m, n, k, kernel=_kid(dt))
    for kid in ig.kernels_for(2 if dt == "i16" else 1):
        _, got = gpu_gemm(A, B, C, m, n, k, kernel=kid)
        assert np.array_equal(got, ref), ig.igemm_kernel_name(kid)


def test_tensor_wrapper_workspace_modes():
    import torch
    ig = _ig()
    m, n, k = 1024, 1100, 1300
    A, B, C = workloads.random_operands("i16", m, n, k, seed=51)
    want = oracle_gemm(A, B, C, m, n, k)
    need = ig.igemm_query_plan(2, m, n, k, kernel=_kid("i16"))["workspace_bytes"]
    for mode in (None, "torch", "none", _workspace(need)):
        Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
        kid = -1 if isinstance(mode, str) and mode == "none" else _kid("i16")
        ig.gemm_i16(Ad, Bd, Cd, kernel=kid, workspace=mode)
        torch.cuda.synchronize()
        assert np.array_equal(Cd.cpu().numpy(), want), str(mode)[:20]


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_explicit_packed_needs_workspace(dt):
    """The library allocates nothing: an explicit packed kernel without a
    workspace is refused before anything is enqueued, eagerly and under
    stream capture (nothing recorded), and C is left untouched."""
    import torch
    ig = _ig()
    m, n, k = 256, 256, 512
    A, B, C = workloads.random_operands(dt, m, n, k, seed=53)
    st, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(dt), workspace=None, check_status=False)
    assert st == ig.IGEMM_EINVAL and np.array_equal(got, C)
    Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
    fn = ig.igemm_i16_ex if dt == "i16" else ig.igemm_i8_ex
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            st = fn(m, n, k, Ad, k, Bd, n, Cd, n, s.cuda_stream, _kid(dt), -1)
            Cd.add_(0)   # keep the captured graph non-empty
    assert st == ig.IGEMM_EINVAL
    g.replay()
    torch.cuda.synchronize()
    assert np.array_equal(Cd.cpu().numpy(), C)


@pytest.mark.parametrize("dt,shape", [("i16", (2048, 2048, 1300)), ("i16", (4096, 1024, 512)),
                                      ("i8", (4096, 4096, 768))])
def test_plain_call_without_workspace(dt, shape):
    """igemm_i16 / igemm_i8 (no workspace) on large shapes, where the _ws
    plan packs or takes the direct kernel: they run a kernel that reads A
    and B in place, bit-exact against the oracle."""
    import torch
    ig = _ig()
    m, n, k = shape
    es = 2 if dt == "i16" else 1
    name = ig.igemm_query_plan(es, m, n, k)["kernel_name"]
    assert "packed" in name or "direct" in name
    A, B, C = workloads.random_operands(dt, m, n, k, seed=57 + m)
    Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
    fn = ig.igemm_i16 if dt == "i16" else ig.igemm_i8
    assert fn(m, n, k, Ad, k, Bd, n, Cd, n) == ig.IGEMM_OK
    torch.cuda.synchronize()
    want = oracle_gemm(A, B, C, m, n, k)
    got = Cd.cpu().numpy()
    assert np.array_equal(got, want), describe_mismatch(got, want)


@pytest.mark.parametrize("dt,shape", [("i16", (300, 520, 1000)), ("i8", (300, 520, 1000)),
                                      ("i8", (512, 384, 768)), ("i16", (130, 200, 33000))])
def test_pack_once_multiply_twice(dt, shape):
    """One pack, two multiplies into different C: both match the oracle
    (int8 512x384x768 reads A in place; int16 k = 33000 runs two chunks)."""
    import torch
    ig = _ig()
    m, n, k = shape
    A, B, C1 = workloads.random_operands(dt, m, n, k, seed=800 + m)
    C2 = workloads.random_operands(dt, m, n, 1, seed=900 + m)[2]
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    P = ig.pack(Ad, Bd)
    del Bd   # B is no longer needed once packed
    torch.cuda.synchronize()
    for Cn in (C1, C2):
        Cd = torch.from_numpy(Cn).cuda()
        ig.gemm_prepacked(P, Cd)
        torch.cuda.synchronize()
        want = oracle_gemm(A, B, Cn, m, n, k)
        got = Cd.cpu().numpy()
        assert np.array_equal(got, want), describe_mismatch(got, want)


def test_prepacked_equals_one_shot_call():
    import torch
    ig = _ig()
    m, n, k = 640, 700, 900
    A, B, C = workloads.random_operands("i16", m, n, k, seed=61)
    Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    C1, C2 = torch.from_numpy(C).cuda(), torch.from_numpy(C).cuda()
    ig.gemm_i16(Ad, Bd, C1, kernel=_kid("i16"))
    ig.gemm_prepacked(ig.pack(Ad, Bd), C2)
    torch.cuda.synchronize()
    assert torch.equal(C1, C2)


@pytest.mark.parametrize("kind", ["raw_handle", "torch_stream"])
def test_wrapper_workspace_on_side_stream(kind):
    """gemm_i16 on a side stream given as a raw HIP handle (or a torch
    stream): the workspace taken from torch's allocator on the current stream
    is recorded on the side stream, so memory allocated and overwritten on
    the current stream right after the call cannot reuse it while the side
    stream's pack and multiply kernels still read it."""
    import torch
    ig = _ig()
    m, n, k = 2048, 2048, 2048
    A, B, C = workloads.random_operands("i16", m, n, k, seed=71)
    Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
    need = ig.igemm_query_plan(2, m, n, k)["workspace_bytes"]
    assert need > 0
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    arg = side.cuda_stream if kind == "raw_handle" else side
    ig.gemm_i16(Ad, Bd, Cd, stream=arg)
    junk = [torch.full((need // 4 + 4096,), -1, dtype=torch.int32, device="cuda")
            for _ in range(3)]
    torch.cuda.synchronize()
    want = oracle_gemm(A, B, C, m, n, k)
    got = Cd.cpu().numpy()
    assert np.array_equal(got, want), describe_mismatch(got, want)
    del junk


# Short k over many tiles: k-tile counts 1 to 9 around the boundaries (the
# ragged tail variants and the zero padding up to a multiple of four tiles),
# ragged m and n.
SHORT_K = [2, 63, 64, 65, 128, 200, 256, 290, 383, 448, 511, 512, 513]


@pytest.mark.parametrize("k", SHORT_K)
def test_packed_int16_short_k_tiles(k):
    m, n = 700, 650
    A, B, C = workloads.random_operands("i16", m, n, k, seed=900 + k)
    _check("i16", A, B, C, m, n, k)


@pytest.mark.parametrize("value", [-32768, 32767])
def test_packed_int16_short_k_extremes(value):
    """Every limb sum at its bound with k = 512 and C nonzero."""
    m, n, k = 200, 130, 512
    A = np.full((m, k), value, np.int16)
    B = np.full((k, n), -value if value > 0 else value, np.int16)
    C = np.full((m, n), -7, np.int32)
    got = _check("i16", A, B, C, m, n, k)
    assert np.all(got == got[0, 0])
