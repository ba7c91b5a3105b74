"""Seeded shape fuzz on the GPU: random m, n, k (including tails that are
not multiples of any tile, k below one k-tile and single rows or columns),
random kernel and k-slice count, misaligned bases and padded leading
dimensions. Every case is compared with the oracle bit for bit."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, gpu_gemm, oracle_gemm, restricted

pytestmark = pytest.mark.gpu


def _cases(n_cases=80, seed=2024):
    import paper_2302_07594_amd as ig
    rng = np.random.default_rng(seed)
    out = []
    # (the direct and small-output kernels take only whole k groups and
    # aligned operands; they have fuzzes of their own below)
    kernels = [k for k in range(ig.igemm_num_kernels())
               if not restricted(ig.igemm_kernel_name(k))]
    for i in range(n_cases):
        dt = "i16" if rng.integers(0, 2) else "i8"
        es = 2 if dt == "i16" else 1
        kid = int(rng.choice([k for k in kernels if (ig.igemm_kernel_name(k).startswith("i16")) == (es == 2)]
                             + [-1]))
        m = int(rng.choice([1, 2, 15, 16, 17, 31, 33, 64, 65, 127, 129, 200, 257, 300]))
        n = int(rng.choice([1, 3, 16, 17, 63, 64, 100, 128, 255, 256, 257, 300]))
        k = int(rng.choice([1, 7, 16, 63, 64, 65, 127, 147, 200, 255, 256, 257, 513, 1000]))
        split = int(rng.choice([-1, -1, 1, 2, 3, 5, 8]))
        offs = tuple(int(x) for x in rng.integers(0, 2, 3) * rng.integers(1, 4, 3))
        pads = tuple(int(x) for x in rng.integers(0, 2, 3) * rng.integers(1, 9, 3))
        out.append((i, dt, kid, m, n, k, split, offs, pads))
    return out


_CASES = _cases()


@pytest.mark.parametrize("case", _CASES, ids=[f"c{c[0]}-{c[1]}-k{c[2]}-{c[3]}x{c[4]}x{c[5]}-s{c[6]}"
                                              for c in _CASES])
def test_fuzz_shape(case):
    i, dt, kid, m, n, k, split, offs, pads = case
    A, B, C = workloads.random_operands(dt, m, n, k, seed=5000 + i, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=kid, split=split, offsets=offs)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


def _direct_cases(n_cases=24, seed=2025):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        dt = "i16" if rng.integers(0, 2) else "i8"
        cols = 8 if dt == "i16" else 16          # one 16-byte chunk of B or C row
        m = int(rng.choice([1, 2, 17, 127, 128, 129, 255, 256, 257, 300, 513]))
        n = int(rng.choice([1, 2, 7, 8, 15, 16, 17, 31, 32])) * cols
        k = int(rng.choice([256, 512, 768, 1280, 33024]))
        pads = tuple(int(x) for x in rng.integers(0, 3, 3) * cols)
        out.append((i, dt, m, n, k, pads))
    return out


_DCASES = _direct_cases()


@pytest.mark.parametrize("case", _DCASES, ids=[f"d{c[0]}-{c[1]}-{c[2]}x{c[3]}x{c[4]}"
                                               for c in _DCASES])
def test_fuzz_direct(case):
    """The direct kernels on random m, n (whole 16-byte column chunks), k
    (whole 256-element groups, one case beyond 32768: two launches) and
    padded leading dimensions of whole 16-byte chunks."""
    import paper_2302_07594_amd as ig
    i, dt, m, n, k, pads = case
    name = "i16_direct_128x128" if dt == "i16" else "i8_direct_256x256"
    kid = [x for x in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(x) == name][0]
    A, B, C = workloads.random_operands(dt, m, n, k, seed=7000 + i, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=kid)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


def _small_cases(n_cases=40, seed=2026):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        m = int(rng.choice([1, 2, 49, 63, 64, 65, 127, 196, 200, 300, 784]))
        n = int(rng.choice([1, 2, 7, 8, 9, 16, 32, 64])) * 8
        k = int(rng.choice([1, 2, 3, 4, 5, 7, 9, 18, 36, 72])) * 64
        split = int(rng.choice([-1, -1, 1, 2, 3, 7, 100]))
        pads = tuple(int(x) for x in rng.integers(0, 3, 3) * 8)
        out.append((i, m, n, k, split, pads))
    return out


_SCASES = _small_cases()


@pytest.mark.parametrize("case", _SCASES, ids=[f"s{c[0]}-{c[1]}x{c[2]}x{c[3]}-s{c[4]}"
                                               for c in _SCASES])
def test_fuzz_small(case):
    """The small-output int16 kernel on random m, n (whole 16-byte column
    chunks), k (whole k-tiles, 1 to 72), k slice requests (a workgroup
    takes at most four k-tiles, so a request of too few slices gets more;
    a short last slice repeats its last tile without multiplying it) and
    padded leading dimensions of whole 16-byte chunks."""
    import paper_2302_07594_amd as ig
    i, m, n, k, split, pads = case
    kid = [x for x in range(ig.igemm_num_kernels())
           if ig.igemm_kernel_name(x) == "i16_small_64x64"][0]
    A, B, C = workloads.random_operands("i16", m, n, k, seed=9000 + i, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=kid, split=split)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


def _ragged_cases(n_cases=40, seed=2027):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        m = int(rng.choice([1, 3, 49, 63, 64, 65, 130, 196, 300, 784]))
        n = int(rng.choice([1, 2, 8, 9, 16, 32, 64])) * 8
        k = int(rng.choice([1, 2, 5, 63, 64, 65, 127, 147, 200, 255, 257, 576, 1000, 1153]))
        split = int(rng.choice([-1, -1, -1, 1, 2, 3, 100]))
        pad_a = int(rng.integers(0, 10))
        off_a = int(rng.choice([0, 1, 2, 3, 5]))
        pads = (pad_a, int(rng.integers(0, 3)) * 8, int(rng.integers(0, 3)))
        extreme = bool(rng.integers(0, 4) == 0)
        out.append((i, m, n, k, split, pads, off_a, extreme))
    return out


_RCASES = _ragged_cases()


@pytest.mark.parametrize("case", _RCASES, ids=[f"r{c[0]}-{c[1]}x{c[2]}x{c[3]}-s{c[4]}-o{c[6]}"
                                               for c in _RCASES])
def test_fuzz_small_ragged(case):
    """The ragged variant of the small-output int16 kernel: rows of A that
    start at any element (base offsets of 0-5 elements, any lda) and k that
    ends inside a k-tile (1 to 1153), with k slice requests, padded C and
    sometimes all-extreme operands; the automatic plan of such a shape is
    checked too."""
    import paper_2302_07594_amd as ig
    i, m, n, k, split, pads, off_a, extreme = case
    kid = [x for x in range(ig.igemm_num_kernels())
           if ig.igemm_kernel_name(x) == "i16_small_64x64"][0]
    A, B, C = workloads.random_operands("i16", m, n, k, seed=9500 + i, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    if extreme:
        A[:, :] = np.where(A < 0, -32768, 32767).astype(np.int16)
        B[:, :] = np.where(B < 0, -32768, 32767).astype(np.int16)
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=kid, split=split, offsets=(off_a, 0, 0))
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    _, got = gpu_gemm(A, B, C, m, n, k, offsets=(off_a, 0, 0))
    assert np.array_equal(got, want), describe_mismatch(got, want)
