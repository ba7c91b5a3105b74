"""GPU parity of the streaming kernels (few rows of A, B streamed once)
against the CPU oracle, bit-exact. int8: the column-per-wave kernel (operands
with rows of whole 16-byte chunks; 4, 8 or 16 k-steps per workgroup in LDS),
its ring variant (any number of k-steps through eight LDS stages) and the
register kernel (other operands), one and two 16-row MFMA blocks, several row
blocks, single-slice (read-add-write) and multi-slice (atomic) plans, k tails,
misaligned operands. int16: the column-per-wave kernel with the limb split in
registers (ragged columns, short last slices, range and limb extremes)."""
import numpy as np
import pytest

import workloads
from gpu_util import describe_mismatch, gpu_gemm, oracle_gemm

pytestmark = pytest.mark.gpu


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _kid():
    ig = _ig()
    return [i for i in range(ig.igemm_num_kernels())
            if ig.igemm_kernel_name(i) == "i8_stream_32x128"][0]


def _check(m, n, k, split=-1, offsets=(0, 0, 0), pads=(0, 0, 0), seed=0):
    A, B, C = workloads.random_operands("i8", m, n, k, seed=seed, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(), split=split, offsets=offsets)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    # padding columns of C are never written
    assert np.array_equal(got[:, n:], C[:, n:])


# k = 3000: 47 k-steps; split s asks for ceil(47 / s) steps per workgroup,
# rounded up to 4, 8, 16 or 32 (32 only for blocks of 16 rows)
@pytest.mark.parametrize("m", [1, 8, 16, 17, 32, 33, 70])
@pytest.mark.parametrize("split", [1, 3, 6, 12, -1])
def test_stream_workgroup_shapes(m, split):
    _check(m, 1000, 3000, split=split, seed=10 * m + split + 5)


# n = 1008 and lda = 3008: rows of A and B whole 16-byte chunks, the last
# column block partial, k = 3000 ending inside a k-step: the column-per-wave kernel (4, 8 or 16 k-steps per workgroup, all in LDS)
@pytest.mark.parametrize("m", [1, 8, 16, 17, 32, 33, 70])
@pytest.mark.parametrize("split", [1, 3, 6, 12, -1])
def test_stream_lds_workgroup_shapes(m, split):
    ig = _ig()
    p = ig.igemm_query_plan(1, m, 1008, 3000, lda=3008, ldb=1008, ldc=1008, kernel=_kid(),
                            split=split)
    # (automatic plans of more than 16 rows over few column blocks take the
    # register kernel's 16-row blocks instead)
    lds = not (split == -1 and m > 16)
    assert p["vec_a"] == 1 and p["vec_b"] == (1 if lds else 0) and p["threads"] == 512
    # (one slice asks for all 47 k-steps in one workgroup: the ring variant)
    assert p["k_chunk"] in ((256, 512, 1024, 3008) if lds else (1024,))
    _check(m, 1008, 3000, split=split, pads=(8, 0, 0), seed=10 * m + split + 7)


# The ring variant of the column-per-wave kernel: more than 16 k-steps per
# workgroup through eight LDS stages (47 steps in one slice, 24 + 23 in two),
# k ending inside a step, a partial column block.
@pytest.mark.parametrize("m", [1, 9, 16, 17, 32, 70])
@pytest.mark.parametrize("split", [1, 2])
def test_stream_ring_workgroup_shapes(m, split):
    ig = _ig()
    p = ig.igemm_query_plan(1, m, 1008, 3000, lda=3008, ldb=1008, ldc=1008, kernel=_kid(),
                            split=split)
    assert p["vec_b"] == 1 and p["k_chunk"] == 64 * -(-47 // split) and p["split"] == split
    _check(m, 1008, 3000, split=split, pads=(8, 0, 0), seed=10 * m + split + 9)


@pytest.mark.parametrize("shape,split", [((5, 128, 1088), 1), ((32, 2064, 8192), 2),
                                         ((3, 4096, 4096), 3), ((24, 640, 1216), 1)])
def test_stream_ring_ranges(shape, split):
    """Step counts that are and are not multiples of the eight stages (17,
    64, 22, 19 steps), plain read-add-write and atomic slices."""
    m, n, k = shape
    _check(m, n, k, split=split, seed=sum(shape) + split)


@pytest.mark.parametrize("value", [-128, 127])
def test_stream_ring_extremes_long_k(value):
    """One slice of 1094 k-steps through the ring."""
    m, n, k = 9, 304, 70000
    A = np.full((m, k), value, np.int8)
    B = np.full((k, n), value, np.int8)
    C = np.zeros((m, n), np.int32)
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid(), split=1)
    assert np.all(got == np.int32(value * value * k))


@pytest.mark.parametrize("shape,pads", [((5, 304, 200), (0, 0, 0)), ((32, 144, 64), (16, 16, 1)),
                                        ((1, 128, 1), (0, 0, 0)), ((17, 2064, 4096), (48, 0, 3))])
def test_stream_lds_single_slice_and_padding(shape, pads):
    """The column-per-wave kernel with k inside one workgroup's range (plain
    read-add-write), short k, padded leading dimensions of whole 16 bytes."""
    m, n, k = shape
    _check(m, n, k, split=1, pads=pads, seed=sum(shape) + 1)


@pytest.mark.parametrize("value", [-128, 127])
def test_stream_lds_extremes_long_k(value):
    m, n, k = 9, 304, 70000
    A = np.full((m, k), value, np.int8)
    B = np.full((k, n), value, np.int8)
    C = np.zeros((m, n), np.int32)
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid())
    assert np.all(got == np.int32(value * value * k))


@pytest.mark.parametrize("shape", [(5, 300, 200), (32, 129, 64), (20, 777, 17), (1, 128, 1)])
def test_stream_single_slice(shape):
    """k within one workgroup's range: one slice, plain read-add-write."""
    ig = _ig()
    m, n, k = shape
    p = ig.igemm_query_plan(1, m, n, k, kernel=_kid())
    assert p["split"] == 1
    _check(m, n, k, seed=sum(shape))


@pytest.mark.parametrize("offsets,pads", [((1, 0, 0), (0, 0, 0)), ((0, 3, 0), (0, 0, 0)),
                                          ((0, 0, 0), (5, 3, 2)), ((2, 1, 1), (1, 7, 3))])
def test_stream_unaligned(offsets, pads):
    """Unaligned A rows or B rows take the byte-load variant."""
    _check(24, 500, 700, offsets=offsets, pads=pads, seed=sum(offsets) + sum(pads))


@pytest.mark.parametrize("value", [-128, 127])
def test_stream_extremes_long_k(value):
    m, n, k = 9, 300, 70000
    A = np.full((m, k), value, np.int8)
    B = np.full((k, n), value, np.int8)
    C = np.zeros((m, n), np.int32)
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid())
    assert np.all(got == np.int32(value * value * k))


@pytest.mark.parametrize("m,n", [(1, 4096), (8, 4096), (32, 4096), (1, 11008), (8, 11008),
                                 (32, 11008)])
def test_stream_inference_shapes(m, n):
    """The weight-streaming shapes (k = 4096) in the launch configuration the
    automatic plan uses."""
    ig = _ig()
    k = 4096
    p = ig.igemm_query_plan(1, m, n, k)
    assert p["kernel_name"] == "i8_stream_32x128"
    A, B, C = workloads.random_operands("i8", m, n, k, seed=m + n)
    _, got = gpu_gemm(A, B, C, m, n, k)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)


# ---------------------------------------------------------------------------
# The int16 column-per-wave kernel (64 columns per workgroup, each element
# split into its two int8 limbs in registers): A and B 16-byte aligned with
# rows of whole 16-byte chunks, k a multiple of 64, n a multiple of 8.

def _kid16():
    ig = _ig()
    return [i for i in range(ig.igemm_num_kernels())
            if ig.igemm_kernel_name(i) == "i16_stream_32x64"][0]


def _check16(m, n, k, split=-1, pads=(0, 0, 0), seed=0):
    A, B, C = workloads.random_operands("i16", m, n, k, seed=seed, lda=k + pads[0],
                                        ldb=n + pads[1], ldc=n + pads[2])
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid16(), split=split)
    want = oracle_gemm(A, B, C, m, n, k)
    assert np.array_equal(got, want), describe_mismatch(got, want)
    assert np.array_equal(got[:, n:], C[:, n:])


# n = 1000: the last of 16 column blocks holds 40 columns; k = 3008: 47
# k-steps, so slices of 4 or 8 steps end with a short one; rows in one or two
# 16-row MFMA blocks and several row blocks
@pytest.mark.parametrize("m", [1, 5, 16, 17, 32, 33, 70])
@pytest.mark.parametrize("split", [1, 6, 12, -1])
def test_stream16_workgroup_shapes(m, split):
    ig = _ig()
    p = ig.igemm_query_plan(2, m, 1000, 3008, lda=3016, ldb=1008, ldc=1003, kernel=_kid16(),
                            split=split)
    assert p["k_chunk"] == (512 if split in (1, 6) else 256) and p["threads"] == 256
    assert p["grid"] == p["tiles"] * p["split"]
    _check16(m, 1000, 3008, split=split, pads=(8, 8, 3), seed=10 * m + split + 11)


@pytest.mark.parametrize("shape", [(3, 64, 64), (32, 8, 128), (20, 520, 512), (9, 136, 576)])
def test_stream16_short_k_and_narrow(shape):
    """One k-step, one workgroup range exactly, a slice of one step, a single
    8-column group."""
    m, n, k = shape
    _check16(m, n, k, seed=sum(shape) + 3)


@pytest.mark.parametrize("va,vb", [(-32768, -32768), (-32768, 32767), (32767, 32767),
                                   (-1, -32768), (255, 256)])
def test_stream16_extremes(va, vb):
    """Constant operands at the int16 range ends and at the limb boundaries:
    C = va * vb * k modulo 2^32, over 140 slices of 512 k."""
    m, n, k = 17, 200, 71680
    A = np.full((m, k), va, np.int16)
    B = np.full((k, n), vb, np.int16)
    C = np.full((m, n), -3, np.int32)
    _, got = gpu_gemm(A, B, C, m, n, k, kernel=_kid16())
    want = (np.int64(va) * vb * k - 3 + (1 << 31)) % (1 << 32) - (1 << 31)
    assert np.all(got == np.int32(want)), (got.min(), got.max(), want)


@pytest.mark.parametrize("m,n", [(1, 4096), (8, 4096), (32, 4096), (1, 11008), (8, 11008),
                                 (32, 11008)])
def test_stream16_inference_shapes(m, n):
    """The weight-streaming shapes with k = 4096, with the kernel asked for
    and in the automatic plan (which takes it up to 16 rows)."""
    ig = _ig()
    k = 4096
    assert (ig.igemm_query_plan(2, m, n, k)["kernel_name"] == "i16_stream_32x64") == (m <= 16)
    A, B, C = workloads.random_operands("i16", m, n, k, seed=m + n + 1)
    want = oracle_gemm(A, B, C, m, n, k)
    for kernel in (_kid16(), -1):
        _, got = gpu_gemm(A, B, C, m, n, k, kernel=kernel)
        assert np.array_equal(got, want), describe_mismatch(got, want)
