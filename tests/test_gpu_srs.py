"""GPU parity of the int16-output update (shift-round-saturate conversion per
k block, the micro-kernel epilogue of the paper) against the oracle, element
by element and bit-exact, through the C ABI."""
import numpy as np
import pytest

import workloads
from gpu_util import to_device

pytestmark = pytest.mark.gpu

SRS_KERNELS = {"i16": ("i16_128x128", "i16_64x64", "i16_32x128", "i16_16x128"),
               "i8": ("i8_32x256", "i8_16x256")}
NP_T = {"i16": np.int16, "i8": np.int8}
SENTINEL = 0x5A5A


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _kid(name):
    ig = _ig()
    return [ig.igemm_kernel_name(i) for i in range(ig.igemm_num_kernels())].index(name)


def _operands(dt, m, n, k, seed, lo=None, hi=None, pad=(0, 0, 0)):
    """A (m x k+pad), B (k x n+pad), C16 (m x n+pad) with padding drawn like
    the data, so stray reads change results and stray writes are visible."""
    t = NP_T[dt]
    info = np.iinfo(t)
    lo = info.min if lo is None else max(lo, info.min)
    hi = info.max if hi is None else min(hi, info.max)
    rng = np.random.default_rng(seed)
    A = rng.integers(lo, hi, size=(m, k + pad[0]), dtype=t, endpoint=True)
    B = rng.integers(lo, hi, size=(k, n + pad[1]), dtype=t, endpoint=True)
    C = rng.integers(-32768, 32767, size=(m, n + pad[2]), dtype=np.int16, endpoint=True)
    return A, B, C


def _oracle(A, B, C, m, n, k, kc, shift, rnd):
    import oracle
    out = C.copy()
    oracle.igemm_srs(A[:m, :k], B[:k, :n], out[:m, :n], kc, shift, rnd)
    return out


def _gpu(A, B, C, m, n, k, kc, shift, rnd, kernel=-1, offsets=(0, 0, 0), check=True,
         workspace=True):
    """igemm_srs_ws with a workspace of the queried size when the plan packs
    the operands (workspace=True), else igemm_srs_ex (no workspace)."""
    import torch
    ig = _ig()
    es = 2 if A.dtype == np.int16 else 1
    Ad = to_device(A, offsets[0])
    Bd = to_device(B, offsets[1])
    Cd = to_device(C, offsets[2])
    args = (es, m, n, k, Ad.data_ptr(), A.shape[1], Bd.data_ptr(), B.shape[1], Cd.data_ptr(),
            C.shape[1], kc)
    need = 0
    if workspace:
        try:
            need = ig.igemm_srs_query(*args, num_cu=torch.cuda.get_device_properties(0)
                                      .multi_processor_count, kernel=kernel)
        except ig.IgemmError:
            need = 0   # the call itself reports the invalid argument
    s = torch.cuda.current_stream().cuda_stream
    if need > 0:
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        st = ig.igemm_srs_ws(*args, shift, 1 if rnd else 0, s, kernel, ws.data_ptr(), need)
    else:
        st = ig.igemm_srs_ex(*args, shift, 1 if rnd else 0, s, kernel)
    torch.cuda.synchronize()
    if check:
        assert st == 0, f"status {st}: {ig.igemm_strerror(st)}"
    return st, Cd.cpu().numpy()


def _describe(got, want, limit=5):
    bad = np.argwhere(got != want)
    lines = [f"{len(bad)} of {got.size} elements differ"]
    for (i, j) in bad[:limit]:
        lines.append(f"  [{i},{j}] got {got[i, j]} want {want[i, j]}")
    return "\n".join(lines)


def _check(A, B, C, m, n, k, kc, shift, rnd, **kw):
    want = _oracle(A, B, C, m, n, k, kc, shift, rnd)
    _, got = _gpu(A, B, C, m, n, k, kc, shift, rnd, **kw)
    assert np.array_equal(got, want), _describe(got, want)
    return got


SHAPES = [(64, 64, 64), (67, 133, 200), (16, 128, 5), (1, 37, 290), (100, 1, 130),
          (33, 257, 700)]
CONVERSIONS = [(0, 0, False), (290, 0, False), (64, 7, True), (100, 12, False), (1, 3, True),
               (0, 20, True), (7, 30, False)]


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_srs_kernel(dt, shape):
    """Every int16-output kernel of the type on ragged shapes, for block
    sizes that do and do not divide k (or exceed it), shifts that saturate
    nearly everything (0) and ones that saturate little, both roundings."""
    m, n, k = shape
    A, B, C = _operands(dt, m, n, k, seed=300 + m + n + k)
    for name in SRS_KERNELS[dt]:
        for kc, shift, rnd in CONVERSIONS:
            _check(A, B, C, m, n, k, kc, shift, rnd, kernel=_kid(name))


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_small_values_reduce_to_gemm(dt):
    """Values small enough that nothing saturates: shift 0 gives C + A B
    exactly, whatever the block size (checked against the plain product)."""
    m, n, k = 150, 140, 200
    A, B, C = _operands(dt, m, n, k, seed=11, lo=-6, hi=6)
    C = (C // 4).astype(np.int16)
    want = (C.astype(np.int64) + A.astype(np.int64) @ B.astype(np.int64)).astype(np.int16)
    for kc in (0, 1, 64, 77, 200):
        _, got = _gpu(A, B, C, m, n, k, kc, 0, False)
        assert np.array_equal(got, want), _describe(got, want)


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("offsets,pad", [((1, 0, 0), (0, 0, 0)), ((0, 1, 1), (0, 0, 0)),
                                         ((0, 0, 0), (3, 5, 7)), ((1, 1, 1), (1, 3, 2))])
def test_alignment_and_padding(dt, offsets, pad):
    """Misaligned bases and odd leading dimensions; padding columns of C
    must be untouched."""
    m, n, k = 90, 150, 300
    A, B, C = _operands(dt, m, n, k, seed=55, pad=pad)
    for name in SRS_KERNELS[dt]:
        got = _check(A, B, C, m, n, k, 100, 9, True, kernel=_kid(name), offsets=offsets)
        assert np.array_equal(got[:, n:], C[:, n:])


def test_extreme_values_and_long_blocks():
    """All-extreme operands: block sums up to 32768 * 2^30 (beyond 2^44),
    exact before the shift; blocks of the maximum length, and a k of two
    maximal blocks plus a tail."""
    m, n = 40, 70
    for k, kc, shift in ((32768, 0, 40), (70000, 32768, 45), (5000, 5000, 0)):
        A = np.full((m, k), -32768, dtype=np.int16)
        B = np.full((k, n), -32768, dtype=np.int16)
        B[:, ::3] = 32767
        A[::5, :] = 32767
        C = np.random.default_rng(k).integers(-32768, 32767, size=(m, n), dtype=np.int16,
                                              endpoint=True)
        for rnd in (False, True):
            _check(A, B, C, m, n, k, kc, shift, rnd)


def test_block_beyond_limit_is_refused():
    m, n, k = 8, 8, 40000
    A, B, C = _operands("i16", m, n, k, seed=2)
    st, got = _gpu(A, B, C, m, n, k, 0, 0, False, check=False)
    assert st == _ig().IGEMM_ENOTSUP and np.array_equal(got, C)


@pytest.mark.parametrize("path", ["packed", "fused"])
def test_paper_shape_full(path):
    """The paper's GEMM shape (4096, 4096, 290) with its k_c = 290 and shift
    0, full-range int16 operands and a random int16 C (the configuration the
    benchmark times): every element against the oracle, on the packed path
    (with a workspace, as the benchmark runs it) and on the fused path (no
    workspace)."""
    case = workloads.WORKLOADS["i16_paper"].cases[0]
    m, n, k = case.m, case.n, case.k
    A, B, _ = workloads.generate(case)
    C = np.random.default_rng(case.seed).integers(-32768, 32767, size=(m, n), dtype=np.int16,
                                                  endpoint=True)
    _, got = _gpu(A, B, C, m, n, k, 290, 0, False, workspace=path == "packed")
    want = _oracle(A, B, C, m, n, k, 290, 0, False)
    assert np.array_equal(got, want), _describe(got, want)


def test_tensor_wrapper_and_graph_replays():
    """gemm_srs() on torch tensors, then captured in a HIP graph (several
    launches, one per block; no workspace, no memset): each replay adds the
    converted blocks once more, checked after every replay."""
    import torch
    ig = _ig()
    m, n, k, kc, shift = 130, 96, 300, 128, 6
    A, B, C = _operands("i16", m, n, k, seed=8, lo=-3000, hi=3000)
    Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
    ig.gemm_srs(Ad, Bd, Cd, kc=kc, shift=shift, round_half_up=True)
    torch.cuda.synchronize()
    want = _oracle(A, B, C, m, n, k, kc, shift, True)
    assert np.array_equal(Cd.cpu().numpy(), want)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ig.gemm_srs(Ad, Bd, Cd, kc=kc, shift=shift, round_half_up=True)
    for rep in range(3):
        g.replay()
        filler = torch.ones(1 << 16, device="cuda", dtype=torch.int32) * rep  # eager work
        torch.cuda.synchronize()
        want = _oracle(A, B, want, m, n, k, kc, shift, True)
        got = Cd.cpu().numpy()
        assert np.array_equal(got, want), f"replay {rep}: " + _describe(got, want)
        del filler


def _fuzz_cases(n_cases=60, seed=777):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        dt = "i16" if rng.integers(0, 3) else "i8"
        m = int(rng.choice([1, 2, 15, 16, 17, 31, 33, 64, 65, 127, 129, 200, 300]))
        n = int(rng.choice([1, 3, 16, 63, 64, 100, 128, 255, 257, 300]))
        k = int(rng.choice([1, 7, 63, 64, 65, 147, 256, 290, 513, 1000]))
        kc = int(rng.choice([0, 0, 1, 5, 64, 100, 256, 290, 2000]))
        shift = int(rng.choice([0, 0, 1, 4, 8, 13, 16, 24, 31, 47]))
        rnd = bool(rng.integers(0, 2))
        kname = str(rng.choice(list(SRS_KERNELS[dt]) + ["auto"]))
        offs = tuple(int(x) for x in rng.integers(0, 2, 3) * rng.integers(1, 4, 3))
        pads = tuple(int(x) for x in rng.integers(0, 2, 3) * rng.integers(1, 9, 3))
        scale = int(rng.choice([8, 300, 0]))  # 0: full range
        out.append((i, dt, m, n, k, kc, shift, rnd, kname, offs, pads, scale))
    return out


_FUZZ = _fuzz_cases()


@pytest.mark.parametrize("case", _FUZZ, ids=[f"f{c[0]}-{c[1]}-{c[2]}x{c[3]}x{c[4]}-kc{c[5]}-s{c[6]}"
                                             for c in _FUZZ])
def test_fuzz_srs(case):
    """Seeded random shapes, block sizes, shifts, roundings, kernels,
    misaligned bases and padded leading dimensions, operand ranges from
    small (nothing saturates) to full."""
    i, dt, m, n, k, kc, shift, rnd, kname, offs, pads, scale = case
    lo, hi = (None, None) if scale == 0 else (-scale, scale)
    A, B, C = _operands(dt, m, n, k, seed=9000 + i, lo=lo, hi=hi, pad=pads)
    kid = -1 if kname == "auto" else _kid(kname)
    _check(A, B, C, m, n, k, kc, shift, rnd, kernel=kid, offsets=offs)


def test_4096_cube_blocks_of_256_full():
    """The benchmark's second int16-output configuration: 4096^3 with
    k_c = 256 (sixteen blocks), full-range operands, random int16 C, on the
    packed path the benchmark times: every element against the oracle."""
    case = workloads.WORKLOADS["i16_4096"].cases[0]
    m, n, k = case.m, case.n, case.k
    A, B, _ = workloads.generate(case)
    C = np.random.default_rng(case.seed).integers(-32768, 32767, size=(m, n), dtype=np.int16,
                                                  endpoint=True)
    _, got = _gpu(A, B, C, m, n, k, 256, 0, False)
    want = _oracle(A, B, C, m, n, k, 256, 0, False)
    assert np.array_equal(got, want), _describe(got, want)


@pytest.mark.parametrize("shape", [(1100, 1030, 700), (128, 128, 256), (257, 300, 1024),
                                   (64, 2000, 290), (200, 150, 350)],
                         ids=lambda s: "x".join(map(str, s)))
def test_packed_kernel(shape):
    """The packed int16 path (operands packed once, exact per-block limb sums
    of the packed planes, one multiply per block): one block and blocks of
    256 / 512, shifts and roundings, ragged shapes. Blocks of 3, 5, 6 and 11
    k-tiles of 64 take the tail chosen at run time, those of 4, 8 and 16 the
    one fixed at build time."""
    m, n, k = shape
    kid = _kid("i16_packed_128x128")
    A, B, C = _operands("i16", m, n, k, seed=600 + m + n + k)
    for kc, shift, rnd in ((0, 0, False), (256, 0, False), (512, 9, True), (k + 5, 20, True),
                           (256, 31, False)):
        _check(A, B, C, m, n, k, kc, shift, rnd, kernel=kid)


@pytest.mark.parametrize("kc", [256, 512, 2048])
def test_packed_multi_block_conversion_forms(kc):
    """The one-launch update of 2-16 whole blocks (k_c <= 2048, shift <= 16)
    converts each block in 32-bit integer arithmetic, in three forms (shift 0,
    1-7, 8-16). Every form with and without rounding, on full-range operands,
    on small operands whose block products straddle the saturation bounds at
    each shift, and on all-extreme operands whose high-limb sums exceed the
    clamp of the conversion (2^21), against the oracle element by element.
    Shifts above 16 and blocks above 2048 take one launch per block."""
    kid = _kid("i16_packed_128x128")
    m, n = 256, 192
    nblk = 16 if kc < 2048 else 3
    k = nblk * kc
    full = _operands("i16", m, n, k, seed=700 + kc)
    small = _operands("i16", m, n, k, seed=701 + kc, lo=-300, hi=300)
    A = np.full((m, k), -32768, dtype=np.int16)
    B = np.full((k, n), -32768, dtype=np.int16)
    B[:, ::3] = 32767
    A[::5, :] = 32767
    A[1::7, : k // 2] = 0      # blocks with zero high-limb sums next to clamped ones
    ext = (A, B, full[2])
    for ops in (full, small, ext):
        for shift in (0, 1, 7, 8, 9, 15, 16, 17):
            for rnd in ((False, True) if shift > 0 else (False,)):
                _check(*ops, m, n, k, kc, shift, rnd, kernel=kid)


def test_packed_kernel_alignment_padding_and_extremes():
    kid = _kid("i16_packed_128x128")
    m, n, k = 300, 260, 768
    A, B, C = _operands("i16", m, n, k, seed=61, pad=(3, 5, 7))
    got = _check(A, B, C, m, n, k, 256, 5, True, kernel=kid, offsets=(1, 1, 1))
    assert np.array_equal(got[:, n:], C[:, n:])
    # one block of 32768 all-extreme elements: sums beyond 2^44, exact
    m, n, k = 130, 140, 32768
    A = np.full((m, k), -32768, dtype=np.int16)
    B = np.full((k, n), -32768, dtype=np.int16)
    B[:, ::3] = 32767
    A[::5, :] = 32767
    C = np.random.default_rng(5).integers(-32768, 32767, size=(m, n), dtype=np.int16,
                                          endpoint=True)
    for shift in (0, 40, 45):
        _check(A, B, C, m, n, k, 0, shift, shift == 45, kernel=kid)


def test_packed_kernel_refuses_unaligned_blocks():
    kid = _kid("i16_packed_128x128")
    A, B, C = _operands("i16", 200, 200, 700, seed=3)
    st, got = _gpu(A, B, C, 200, 200, 700, 100, 0, False, kernel=kid, check=False)
    assert st == _ig().IGEMM_EINVAL and np.array_equal(got, C)


# ---- caller-owned workspace (igemm_srs_ws / igemm_srs_query) ------------------

def _ws_tensor(nbytes, fill=0x5A):
    import torch
    raw = torch.full((nbytes + 512,), fill, dtype=torch.uint8, device="cuda")
    off = (-raw.data_ptr()) % 256
    return raw, raw[off:off + nbytes]


def _srs_ws(A, B, C, m, n, k, kc, shift, rnd, ws, ws_bytes, kernel=-1, ws_ptr=None):
    import torch
    ig = _ig()
    es = 2 if A.dtype == np.int16 else 1
    Ad, Bd, Cd = (torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (A, B, C))
    ptr = ws_ptr if ws_ptr is not None else (ws.data_ptr() if ws is not None else None)
    st = ig.igemm_srs_ws(es, m, n, k, Ad.data_ptr(), A.shape[1], Bd.data_ptr(), B.shape[1],
                         Cd.data_ptr(), C.shape[1], kc, shift, 1 if rnd else 0,
                         torch.cuda.current_stream().cuda_stream, kernel, ptr, ws_bytes)
    torch.cuda.synchronize()
    return st, Cd.cpu().numpy()


def _num_cu():
    import torch
    return torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("shape,kc", [((1100, 1030, 700), 256), ((1100, 1030, 700), 0),
                                      ((64, 2000, 290), 0), ((2048, 1024, 1024), 512)],
                         ids=["1100x1030x700-kc256", "1100x1030x700-kc0", "64x2000x290-kc0",
                              "2048x1024x1024-kc512"])
def test_ws_packed_path_matches_oracle(shape, kc):
    """A caller's workspace (stale contents) holds the packed operands and the
    limb sums; the result is the oracle's, bit for bit."""
    ig = _ig()
    m, n, k = shape
    A, B, C = _operands("i16", m, n, k, seed=900 + m + k + kc)
    kid = _kid("i16_packed_128x128")
    need = ig.igemm_srs_query(2, m, n, k, 1 << 20, k, 1 << 20, n, 1 << 20, n, kc, _num_cu(), kid)
    assert need > 0
    _, ws = _ws_tensor(need)
    want = _oracle(A, B, C, m, n, k, kc, 7, True)
    st, got = _srs_ws(A, B, C, m, n, k, kc, 7, True, ws, need, kernel=kid)
    assert st == 0 and np.array_equal(got, want), _describe(got, want)


def test_ws_auto_choice_and_errors():
    """Automatic choice with the queried workspace; too small a workspace is
    ENOMEM and a misaligned one EINVAL, both with C unchanged; a fused choice
    needs no workspace."""
    ig = _ig()
    m, n, k, kc = 4096, 1024, 512, 256
    A, B, C = _operands("i16", m, n, k, seed=91)
    need = ig.igemm_srs_query(2, m, n, k, 1 << 20, k, 1 << 20, n, 1 << 20, n, kc, _num_cu())
    assert need > 0
    raw, ws = _ws_tensor(need)
    want = _oracle(A, B, C, m, n, k, kc, 0, False)
    st, got = _srs_ws(A, B, C, m, n, k, kc, 0, False, ws, need)
    assert st == 0 and np.array_equal(got, want), _describe(got, want)
    st, got = _srs_ws(A, B, C, m, n, k, kc, 0, False, ws, need - 1)
    assert st == ig.IGEMM_ENOMEM and np.array_equal(got, C)
    st, got = _srs_ws(A, B, C, m, n, k, kc, 0, False, None, need, ws_ptr=ws.data_ptr() + 16)
    assert st == ig.IGEMM_EINVAL and np.array_equal(got, C)
    # int8 operands, and blocks of 100: fused, no workspace needed or touched
    for dt, kc2 in (("i8", 256), ("i16", 100)):
        A2, B2, C2 = _operands(dt, 300, 200, 700, seed=92)
        es = 2 if dt == "i16" else 1
        assert ig.igemm_srs_query(es, 300, 200, 700, 1 << 20, 700, 1 << 20, 200, 1 << 20, 200,
                                  kc2, _num_cu()) == 0
        want = _oracle(A2, B2, C2, 300, 200, 700, kc2, 3, False)
        st, got = _srs_ws(A2, B2, C2, 300, 200, 700, kc2, 3, False, None, 0)
        assert st == 0 and np.array_equal(got, want), _describe(got, want)


def test_ws_packed_path_in_graph():
    """gemm_srs with its default workspace (torch's allocator) captured into
    a graph on a shape that takes the packed path: every replay, with eager
    work between them, gives the oracle's result."""
    import torch
    ig = _ig()
    m, n, k, kc, shift = 4096, 1024, 768, 256, 4
    assert ig.igemm_srs_query(2, m, n, k, 1 << 20, k, 1 << 20, n, 1 << 20, n, kc, _num_cu()) > 0
    A, B, C = _operands("i16", m, n, k, seed=93)
    want = _oracle(A, B, C, m, n, k, kc, shift, False)
    Ad, Bd, C0 = (torch.from_numpy(x).cuda() for x in (A, B, C))
    Cd = C0.clone()
    ig.gemm_srs(Ad, Bd, Cd, kc=kc, shift=shift)
    torch.cuda.synchronize()
    assert np.array_equal(Cd.cpu().numpy(), want)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        Cd.copy_(C0)
        ig.gemm_srs(Ad, Bd, Cd, kc=kc, shift=shift)
    for rep in range(3):
        Cd.fill_(rep + 1)
        g.replay()
        filler = torch.ones(1 << 16, device="cuda", dtype=torch.int32) * rep  # eager work
        torch.cuda.synchronize()
        got = Cd.cpu().numpy()
        assert np.array_equal(got, want), f"replay {rep}: " + _describe(got, want)
        del filler
