"""GPU parity: the HIP path (through the C ABI) against the CPU oracle,
element by element and bit-exact (integer arithmetic modulo 2^32 has a
unique result, so there is no tolerance)."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, general_kernels, gpu_gemm, oracle_gemm

pytestmark = pytest.mark.gpu

NP_T = {"i16": np.int16, "i8": np.int8}


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _check(A, B, C, m, n, k, **kw):
    _, got = gpu_gemm(A, B, C, m, n, k, **kw)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    return got


def test_int16_256_cube_full():
    """int16 m=n=k=256, full-range operands, C zero, seed 0."""
    case = workloads.WORKLOADS["i16_256"].cases[0]
    A, B, C = workloads.generate(case)
    _check(A, B, C, case.m, case.n, case.k)


def _kernel_shapes(name):
    bm, bn = (int(x) for x in name.split("_")[-1].split("x"))
    if "small" in name:
        # k a multiple of 64, n a multiple of 8 columns; m, n ragged
        return [
            (bm, bn, 64),                      # exactly one tile, one k-tile
            (bm + 3, bn + 8, 320),             # ragged m and n, five k-tiles
            (2 * bm - 1, 2 * bn + 8, 1024),    # several tiles, k sliced
            (1, bn - 8, 64 * 9),               # one row, a short last slice
            (bm - 1, 8, 256),                  # eight columns
        ]
    if "i16_stream" in name:
        # k a multiple of 64, n a multiple of 8 columns; m, n ragged
        return [
            (bm, bn, 64),                      # exactly one block, one k-step
            (bm + 3, bn + 8, 320),             # ragged m and n, five k-steps
            (2 * bm - 1, 2 * bn + 8, 1024),    # several blocks, k sliced
            (1, bn - 8, 64 * 9),               # one row, a short last slice
            (bm - 1, 8, 256),                  # eight columns
        ]
    if "direct" in name:
        # k a multiple of 256, n a multiple of 16 columns; m, n ragged
        return [
            (bm, bn, 256),                     # exactly one tile, four k-tiles
            (bm + 3, bn + 16, 768),            # ragged m and n, several tiles
            (2 * bm - 1, 2 * bn + 16, 512),
            (1, bn - 16, 256),                 # one row
            (bm - 1, 16, 1024),                # sixteen columns
        ]
    return [
        (bm, bn, 64),                      # exactly one tile, one k-tile
        (bm + 3, bn + 5, 3 * 64 + 17),     # ragged m, n and k tails, several tiles
        (2 * bm - 1, 2 * bn + 1, 5),       # k smaller than one k-tile
        (1, bn - 7, 130),                  # one row
        (bm - 1, 1, 200),                  # one column
    ]


def _kernel_cases():
    ig = _ig()
    out = []
    for kid in range(ig.igemm_num_kernels()):
        name = ig.igemm_kernel_name(kid)
        for shape in _kernel_shapes(name):
            for split in (-1, 1, 3):
                out.append((kid, name, shape, split))
    return out


_KCASES = _kernel_cases()


@pytest.mark.parametrize("kid,name,shape,split", _KCASES,
                         ids=[f"{c[1]}-{'x'.join(map(str, c[2]))}-s{c[3]}" for c in _KCASES])
def test_every_kernel_ragged(kid, name, shape, split):
    dt = "i16" if name.startswith("i16") else "i8"
    m, n, k = shape
    A, B, C = workloads.random_operands(dt, m, n, k, seed=1000 + kid * 7 + m + n + k)
    _check(A, B, C, m, n, k, kernel=kid, split=split)


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("offsets,pad", [((0, 0, 0), (0, 0, 0)), ((1, 0, 0), (0, 0, 0)),
                                         ((0, 1, 0), (0, 0, 0)), ((0, 0, 1), (0, 0, 0)),
                                         ((0, 0, 0), (3, 5, 7)), ((1, 1, 1), (1, 3, 2))])
def test_alignment_and_padding(dt, offsets, pad):
    """Misaligned bases and odd leading dimensions take the element path;
    padding columns of C (sentinels) must be untouched."""
    m, n, k = 150, 140, 200
    A, B, C = workloads.random_operands(dt, m, n, k, seed=77, lda=k + pad[0], ldb=n + pad[1],
                                        ldc=n + pad[2])
    for kid in general_kernels(2 if dt == "i16" else 1):
        got = _check(A, B, C, m, n, k, kernel=kid, offsets=offsets)
        assert np.array_equal(got[:, n:], C[:, n:])


@pytest.mark.parametrize("value", [-32768, 32767])
@pytest.mark.parametrize("k", [4096, 40000])
def test_int16_extremes_and_long_k(value, k):
    """Constant extreme operands: every limb sum is at its bound; k = 40000
    exceeds the per-workgroup k range, so slices are added atomically."""
    m, n = 40, 70
    A = np.full((m, k), value, np.int16)
    B = np.full((k, n), value, np.int16)
    C = np.zeros((m, n), np.int32)
    got = _check(A, B, C, m, n, k)
    assert np.all(got == got[0, 0])


@pytest.mark.parametrize("value", [-128, 127])
def test_int8_extremes_long_k(value):
    m, n, k = 33, 65, 70000
    A = np.full((m, k), value, np.int8)
    B = np.full((k, n), value, np.int8)
    C = np.full((m, n), 2 ** 31 - 1000, np.int32)
    _check(A, B, C, m, n, k)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_deterministic_with_slices(dt):
    m, n, k = 97, 301, 2000
    A, B, C = workloads.random_operands(dt, m, n, k, seed=5)
    _, g1 = gpu_gemm(A, B, C, m, n, k, split=7)
    _, g2 = gpu_gemm(A, B, C, m, n, k, split=7)
    _, g3 = gpu_gemm(A, B, C, m, n, k, split=1)
    assert np.array_equal(g1, g2) and np.array_equal(g1, g3)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_degenerate_sizes_on_device(dt):
    ig = _ig()
    import torch
    C = torch.arange(12, dtype=torch.int32, device="cuda").reshape(3, 4)
    before = C.clone()
    A = torch.zeros((3, 1), dtype=getattr(torch, "int16" if dt == "i16" else "int8"),
                    device="cuda")
    fn = ig.igemm_i16 if dt == "i16" else ig.igemm_i8
    s = torch.cuda.current_stream().cuda_stream
    assert fn(3, 4, 0, A.data_ptr(), 1, A.data_ptr(), 4, C.data_ptr(), 4, s) == 0   # k = 0
    assert fn(0, 4, 1, A.data_ptr(), 1, A.data_ptr(), 4, C.data_ptr(), 4, s) == 0   # m = 0
    assert fn(3, 0, 1, A.data_ptr(), 1, A.data_ptr(), 4, C.data_ptr(), 4, s) == 0   # n = 0
    torch.cuda.synchronize()
    assert torch.equal(C, before)


@pytest.mark.parametrize("dt", ["i16", "i8"])
def test_column_major_via_transpose_identity(dt):
    """A column-major caller passes (n, m, k, B, A): C^T += B^T A^T."""
    m, n, k = 70, 90, 150
    A, B, C = workloads.random_operands(dt, m, n, k, seed=21)
    # Column-major storage of A (m x k) is row-major storage of A^T (k x m).
    At = np.ascontiguousarray(A.T)   # k x m row-major == A column-major
    Bt = np.ascontiguousarray(B.T)   # n x k row-major == B column-major
    Ct = np.ascontiguousarray(C.T)   # n x m row-major == C column-major
    _, got_t = gpu_gemm(Bt, At, Ct, n, m, k)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got_t.T, want)


def test_nondefault_stream():
    import torch
    ig = _ig()
    m, n, k = 130, 129, 257
    A, B, C = workloads.random_operands("i16", m, n, k, seed=9)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Ad, Bd, Cd = (torch.from_numpy(x).cuda() for x in (A, B, C))
        ig.gemm_i16(Ad, Bd, Cd)
    s.synchronize()
    assert np.array_equal(Cd.cpu().numpy(), oracle_gemm(A, B, C, m, n, k))


def test_tensor_wrappers_reject_bad_inputs():
    import torch
    ig = _ig()
    a = torch.zeros((4, 4), dtype=torch.int16, device="cuda")
    c = torch.zeros((4, 4), dtype=torch.int32, device="cuda")
    with pytest.raises(TypeError):
        ig.gemm_i16(a.to(torch.int8), a, c)
    with pytest.raises(ValueError):
        ig.gemm_i16(a, a[:3], c)
    with pytest.raises(ValueError):
        ig.gemm_i16(a.t(), a, c)  # stride (1, 4): rows are not contiguous


@pytest.mark.parametrize("i", range(len(workloads.CONV_SHAPES)))
def test_conv_shaped_int16_set(i):
    case = workloads.WORKLOADS["i16_conv"].cases[i]
    A, B, C = workloads.generate(case)
    _check(A, B, C, case.m, case.n, case.k)


@pytest.mark.parametrize("i", range(len(workloads.SKINNY_SHAPES)))
def test_skinny_int8_set(i):
    case = workloads.WORKLOADS["i8_skinny"].cases[i]
    A, B, C = workloads.generate(case)
    _check(A, B, C, case.m, case.n, case.k)


@pytest.mark.parametrize("i", range(len(workloads.SKINNY_SHAPES)))
def test_skinny_int16_set(i):
    case = workloads.WORKLOADS["i16_skinny"].cases[i]
    A, B, C = workloads.generate(case)
    _check(A, B, C, case.m, case.n, case.k)


def _full_size(wname):
    """Full-size run of a benchmark workload on both paths: with a workspace
    (the packed plan the benchmark times through the tensor wrappers) and
    without one (igemm_i16 / igemm_i8: in-place kernels). Every element of
    both results is compared with the oracle's."""
    case = workloads.WORKLOADS[wname].cases[0]
    A, B, C = workloads.generate(case)
    m, n, k = case.m, case.n, case.k
    want = oracle_gemm(A, B, C, m, n, k)
    for ws in ("auto", None):
        _, got = gpu_gemm(A, B, C, m, n, k, workspace=ws)
        assert np.array_equal(got, want), f"workspace={ws}: " + describe_mismatch(got, want)
        del got


def test_paper_shape_int16_full():
    """The paper's GEMM shape (4096, 4096, 290), int16, every element."""
    case = workloads.WORKLOADS["i16_paper"].cases[0]
    A, B, C = workloads.generate(case)
    _check(A, B, C, case.m, case.n, case.k)


@pytest.mark.parametrize("name", ["i16_direct_128x128", "i8_direct_256x256", "i16_small_64x64"])
def test_direct_kernel_preconditions(name):
    """The direct kernels take k a multiple of 256, 16-byte aligned operands
    with rows of whole 16 bytes and n a multiple of 16 bytes of columns; an
    explicit request outside that is refused, C untouched. The small-output
    kernel needs this of B only: its ragged variant takes A at any alignment
    and any k (checked against the oracle here)."""
    ig = _ig()
    kid = [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == name][0]
    dt = "i16" if name.startswith("i16") else "i8"
    small = name == "i16_small_64x64"
    for (m, n, k, offs) in ((64, 64, 300 if "direct" in name else 100, (0, 0, 0)),
                            (64, 64, 256, (1, 0, 0)),
                            (64, 64, 256, (0, 1, 0)), (64, 72 if dt == "i8" else 68, 256, (0, 0, 0))):
        A, B, C = workloads.random_operands(dt, m, n, k, seed=77 + k)
        st, got = gpu_gemm(A, B, C, m, n, k, kernel=kid, offsets=offs, check_status=False,
                           workspace=None)
        if small and offs[1] == 0 and n % 8 == 0:
            want = oracle_gemm(A, B, C, m, n, k)
            assert st == 0 and np.array_equal(got, want), (m, n, k, offs)
        else:
            assert st == ig.IGEMM_EINVAL and np.array_equal(got, C), (m, n, k, offs)


def test_int16_4096_cube_full():
    """int16 m=n=k=4096, full-range operands, C uniform in +-2^20, seed 1."""
    _full_size("i16_4096")


def test_int8_8192_cube_full():
    """int8 m=n=k=8192, operands uniform in [-128, 127], C zero, seed 2."""
    _full_size("i8_8192")
