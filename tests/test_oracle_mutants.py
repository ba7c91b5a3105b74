"""Plant plausible mistakes in copies of the oracle (on the CPU) and check
that the pins catch every one of them. This is evidence that the pins are
strong enough to trust the oracle, not a test of the GPU path."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle_pins as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "igemm_oracle.c")

# (name, text to find, replacement). Each applies to both entry points.
MUTANTS = [
    ("transposed_B", "const int16_t *brow = B + p * ldb;",
     "const int16_t *brow = B + p;"),
    ("transposed_B_i8", "acc[j] += a * (int64_t)brow[j];",
     "acc[j] += a * (int64_t)B[j * ldb + p];"),
    ("dropped_C0", "acc[j] = (int64_t)C[i * ldc + j];", "acc[j] = 0;"),
    ("wrong_sign", "acc[j] += a * (int64_t)brow[j];", "acc[j] -= a * (int64_t)brow[j];"),
    ("k_off_by_one", "for (int64_t p = 0; p < k; ++p)", "for (int64_t p = 1; p < k; ++p)"),
    ("lda_for_ldb", "B + p * ldb", "B + p * lda"),
    ("ldc_as_n", "C[i * ldc + j] = wrap_to_i32", "C[i * n + j] = wrap_to_i32"),
    ("saturate", "if (u <= 0x7FFFFFFFu)\n        return (int32_t)u;",
     "if (v > 2147483647) return 2147483647; if (v < -2147483647 - 1) return -2147483647 - 1;\n"
     "    if (u <= 0x7FFFFFFFu)\n        return (int32_t)u;"),
    ("i16_product_truncated", "acc[j] += a * (int64_t)brow[j];",
     "acc[j] += (int16_t)(a * (int64_t)brow[j]);"),
    ("row_index_for_a", "const int64_t a = (int64_t)A[i * lda + p];",
     "const int64_t a = (int64_t)A[p * lda + i];"),
]


def _build(tmp_path, name, find, repl):
    text = open(SRC).read()
    assert find in text, name
    text = text.replace(find, repl)
    src = tmp_path / f"{name}.c"
    src.write_text(text)
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fopenmp", "-fPIC", "-shared", str(src),
                    "-o", str(lib)], check=True)
    return str(lib)


def _gemm_from(lib_path):
    lib = ctypes.CDLL(lib_path)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    for nm in ("oracle_igemm_i16", "oracle_igemm_i8"):
        getattr(lib, nm).argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64]
        getattr(lib, nm).restype = ctypes.c_int

    def gemm(A, B, C):
        fn = lib.oracle_igemm_i16 if A.dtype == np.int16 else lib.oracle_igemm_i8
        m, k = A.shape
        n = B.shape[1]
        ld = lambda x: x.strides[0] // x.itemsize if x.shape[0] > 0 else max(x.shape[1], 1)
        st = fn(m, n, k, A.ctypes.data_as(vp), ld(A), B.ctypes.data_as(vp), ld(B),
                C.ctypes.data_as(vp), ld(C))
        if st != 0:
            raise AssertionError(f"status {st}")
        return C
    return gemm


@pytest.mark.parametrize("mut", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_mutant(tmp_path, mut):
    name, find, repl = mut
    gemm = _gemm_from(_build(tmp_path, name, find, repl))
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(gemm)
        except AssertionError:
            caught.append(pin.__name__)
        except Exception as e:  # crashes count as caught too, but say so
            caught.append(f"{pin.__name__}:{type(e).__name__}")
    assert caught, f"mutant {name} passed every pin"


def test_unmodified_copy_passes_every_pin(tmp_path):
    gemm = _gemm_from(_build(tmp_path, "unmodified", "static int32_t wrap_to_i32",
                             "static int32_t wrap_to_i32"))
    for pin in pins.ALL_PINS:
        pin(gemm)
