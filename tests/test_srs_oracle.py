"""The int16-output (shift-round-saturate) oracle against its pins, and
plausible mistakes planted in copies of it (on the CPU), each of which some
pin must catch."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import srs_pins as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "igemm_oracle.c")


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_srs_pin(pin):
    pin(oracle.igemm_srs)


def test_oracle_srs_rejects_bad_arguments():
    A = np.zeros((2, 3), np.int16)
    B = np.zeros((3, 2), np.int16)
    C = np.zeros((2, 2), np.int16)
    for kc, shift in ((-1, 0), (0, -1), (0, 48)):
        with pytest.raises(RuntimeError):
            oracle.igemm_srs(A, B, C, kc, shift)
    with pytest.raises(TypeError):
        oracle.igemm_srs(A, B, np.zeros((2, 2), np.int32))


MUTANTS = [
    ("truncate_toward_zero", "    if (v % d != 0 && v < 0)\n        q -= 1;\n", "\n"),
    ("no_upper_saturation", "if (t > 32767)                                                            \\\n"
     "                        t = 32767;", "if (0)                                                                    \\\n"
     "                        t = 32767;"),
    ("saturating_add", "c = (int64_t)wrap_to_i16(c + t);",
     "c = c + t > 32767 ? 32767 : (c + t < -32768 ? -32768 : c + t);"),
    ("blocks_ignored", "const int64_t blk = kc == 0 ? k : kc;", "const int64_t blk = k;"),
    ("round_always", "(round_half_up && shift > 0)", "(shift > 0)"),
    ("round_full_step", "((int64_t)1 << (shift - 1)) : 0;", "((int64_t)1 << shift) : 0;"),
    ("dropped_C0", "int64_t c = (int64_t)C[i * ldc + j];", "int64_t c = 0;"),
    ("block_restarts_at_zero", "for (int64_t p = p0; p < p1; ++p)", "for (int64_t p = 0; p < p1; ++p)"),
]


def _srs_from(tmp_path, name, find, repl):
    text = open(SRC).read()
    assert find in text, name
    src = tmp_path / f"{name}.c"
    src.write_text(text.replace(find, repl))
    lib_path = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fopenmp", "-fPIC", "-shared", str(src), "-o",
                    str(lib_path)], check=True)
    lib = ctypes.CDLL(str(lib_path))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    for nm in ("oracle_igemm_srs_i16", "oracle_igemm_srs_i8"):
        getattr(lib, nm).argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64, i64,
                                     ctypes.c_int, ctypes.c_int]
        getattr(lib, nm).restype = ctypes.c_int

    def srs(A, B, C, kc=0, shift=0, rnd=False):
        A = np.ascontiguousarray(A)
        B = np.ascontiguousarray(B)
        m, k = A.shape
        n = B.shape[1]
        fn = lib.oracle_igemm_srs_i16 if A.dtype == np.int16 else lib.oracle_igemm_srs_i8
        st = fn(m, n, k, A.ctypes.data_as(vp), max(k, 1), B.ctypes.data_as(vp), max(n, 1),
                C.ctypes.data_as(vp), max(n, 1), kc, shift, 1 if rnd else 0)
        if st != 0:
            raise AssertionError(f"status {st}")
        return C
    return srs


@pytest.mark.parametrize("mut", MUTANTS, ids=lambda m: m[0])
def test_srs_pins_catch_mutant(tmp_path, mut):
    name, find, repl = mut
    srs = _srs_from(tmp_path, name, find, repl)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(srs)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"


def test_unmodified_srs_copy_passes_every_pin(tmp_path):
    srs = _srs_from(tmp_path, "unmodified", "int16_t", "int16_t")
    for pin in pins.ALL_PINS:
        pin(srs)
