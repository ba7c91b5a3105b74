"""CPU oracle for integer GEMM C += A.B and for the convolution Y += conv(X, W)
that the lowering of Sec. 4.2 turns into one GEMM -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The GPU library does not depend on it
and must never fall back to it.

The arithmetic lives in ``igemm_oracle.c`` (plain int64 triple loop, reduced
modulo 2^32 at the end; Sec. 4.1 definition of C += A B; the direct
definition of a zero-padded, strided, dilated 2-D convolution in NHWC / filter
row x filter column x input channel x output channel layouts; and the int16
output of the micro-kernel of Sec. 5.2, converted per k_c block by
shift-round-saturate and added with wraparound). This module only marshals
numpy arrays into that library with ctypes.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # IGEMM_ORACLE_LIB names another build of the same source (the sanitizer
    # test loads the copy built with -fsanitize=address,undefined).
    path = os.environ.get("IGEMM_ORACLE_LIB") or _build.LIB
    if path == _build.LIB and not os.path.exists(path):
        _build.build()
    lib = ctypes.CDLL(path)
    i64 = ctypes.c_int64
    vp = ctypes.c_void_p
    for name in ("oracle_igemm_i16", "oracle_igemm_i8"):
        fn = getattr(lib, name)
        fn.argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64]
        fn.restype = ctypes.c_int
    for name in ("oracle_conv2d_i16", "oracle_conv2d_i8"):
        fn = getattr(lib, name)
        fn.argtypes = [i64] * 13 + [vp, vp, vp]
        fn.restype = ctypes.c_int
    for name in ("oracle_igemm_srs_i16", "oracle_igemm_srs_i8"):
        fn = getattr(lib, name)
        fn.argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64, i64, ctypes.c_int,
                       ctypes.c_int]
        fn.restype = ctypes.c_int
    lib.oracle_conv2d_out_dim.argtypes = [i64] * 5
    lib.oracle_conv2d_out_dim.restype = i64
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def num_threads() -> int:
    """Threads the oracle's OpenMP loop uses."""
    return int(_load().oracle_num_threads())


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _ld(a: np.ndarray, what: str) -> int:
    if a.ndim != 2:
        raise ValueError(f"{what} must be 2-D")
    if a.size == 0:
        return max(a.shape[1], 1)
    if a.shape[1] > 1 and a.strides[1] != a.itemsize:
        raise ValueError(f"{what} must have unit stride along its rows")
    if a.shape[0] == 1:
        return max(a.shape[1], 1)
    return a.strides[0] // a.itemsize


def igemm_raw(dtype: str, m: int, n: int, k: int, A, lda: int, B, ldb: int,
              C, ldc: int) -> int:
    """Call the oracle on raw buffers (numpy arrays used for their memory).

    ``C`` is updated in place. Returns the oracle's status (0 = OK).
    """
    lib = _load()
    fn = lib.oracle_igemm_i16 if dtype == "i16" else lib.oracle_igemm_i8
    return int(fn(m, n, k, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc))


def igemm(A: np.ndarray, B: np.ndarray, C: np.ndarray) -> np.ndarray:
    """C += A.B (mod 2^32) in place on numpy views; returns C.

    A (m x k) and B (k x n) are int16 or int8 (same type); C is int32 m x n.
    Views with a row stride larger than their width are allowed; elements
    outside the views are not touched.
    """
    if A.dtype != B.dtype or A.dtype not in (np.int16, np.int8):
        raise TypeError("A and B must both be int16 or both int8")
    if C.dtype != np.int32:
        raise TypeError("C must be int32")
    m, k = A.shape
    k2, n = B.shape
    if k2 != k or C.shape != (m, n):
        raise ValueError("shape mismatch")
    dtype = "i16" if A.dtype == np.int16 else "i8"
    st = igemm_raw(dtype, m, n, k, A, _ld(A, "A"), B, _ld(B, "B"), C, _ld(C, "C"))
    if st != 0:
        raise RuntimeError(f"oracle returned {st}")
    return C


def conv2d_out_dim(size: int, f: int, stride: int = 1, pad: int = 0, dil: int = 1) -> int:
    """Output extent of one spatial dimension (floor rule; -1 if invalid)."""
    return int(_load().oracle_conv2d_out_dim(size, f, stride, pad, dil))


def conv2d(X: np.ndarray, W: np.ndarray, Y: np.ndarray, stride=(1, 1), pad=(0, 0),
           dil=(1, 1)) -> np.ndarray:
    """Y += conv(X, W) (mod 2^32) in place; returns Y.

    X: n x h x w x c (int16 or int8), W: r x s x c x k (same type),
    Y: n x oh x ow x k int32; all C-contiguous. Zero padding, strides and
    dilations per (height, width).
    """
    if X.dtype != W.dtype or X.dtype not in (np.int16, np.int8):
        raise TypeError("X and W must both be int16 or both int8")
    if Y.dtype != np.int32:
        raise TypeError("Y must be int32")
    for a, nm in ((X, "X"), (W, "W"), (Y, "Y")):
        if a.ndim != 4 or not a.flags.c_contiguous:
            raise ValueError(f"{nm} must be a C-contiguous 4-D array")
    n, h, w, c = X.shape
    r, s, c2, k = W.shape
    oh = conv2d_out_dim(h, r, stride[0], pad[0], dil[0])
    ow = conv2d_out_dim(w, s, stride[1], pad[1], dil[1])
    if c2 != c or Y.shape != (n, oh, ow, k):
        raise ValueError(f"shape mismatch: X {X.shape} W {W.shape} Y {Y.shape}, "
                         f"expected Y {(n, oh, ow, k)}")
    lib = _load()
    fn = lib.oracle_conv2d_i16 if X.dtype == np.int16 else lib.oracle_conv2d_i8
    st = int(fn(n, h, w, c, k, r, s, stride[0], stride[1], pad[0], pad[1], dil[0], dil[1],
                _ptr(X), _ptr(W), _ptr(Y)))
    if st != 0:
        raise RuntimeError(f"oracle returned {st}")
    return Y


def igemm_srs(A: np.ndarray, B: np.ndarray, C: np.ndarray, kc: int = 0, shift: int = 0,
              round_half_up: bool = False) -> np.ndarray:
    """int16-output update in place on numpy views; returns C.

    For each block of kc consecutive k indices (kc = 0: all of k), the exact
    partial product is shifted right by ``shift`` (floor; with round_half_up
    2^(shift-1) is added first), saturated to int16 and added into the int16
    C modulo 2^16. A, B int16 or int8 (same type).
    """
    if A.dtype != B.dtype or A.dtype not in (np.int16, np.int8):
        raise TypeError("A and B must both be int16 or both int8")
    if C.dtype != np.int16:
        raise TypeError("C must be int16")
    m, k = A.shape
    k2, n = B.shape
    if k2 != k or C.shape != (m, n):
        raise ValueError("shape mismatch")
    lib = _load()
    fn = lib.oracle_igemm_srs_i16 if A.dtype == np.int16 else lib.oracle_igemm_srs_i8
    st = int(fn(m, n, k, _ptr(A), _ld(A, "A"), _ptr(B), _ld(B, "B"), _ptr(C), _ld(C, "C"),
                int(kc), int(shift), 1 if round_half_up else 0))
    if st != 0:
        raise RuntimeError(f"oracle returned {st}")
    return C
