"""Seeded shape fuzz on the GPU: random m, n, k (including tails that are
not multiples of any tile, k below one k-tile and single rows or columns),
random kernel and k-slice count, misaligned bases and padded leading
dimensions. Every case is compared with the oracle bit for bit."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, gpu_gemm, oracle_gemm

pytestmark = pytest.mark.gpu


def _cases(n_cases=80, seed=2024):
    import paper_2302_07594_amd as ig
    rng = np.random.default_rng(seed)
    out = []
    kernels = list(range(ig.igemm_num_kernels()))
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
