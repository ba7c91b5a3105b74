"""Pins for the CPU oracle: facts fixed by the paper's definition and by
mathematics, none of which re-types the oracle's own loop.

Each ``pin_*`` function takes ``gemm(A, B, C)`` -- an in-place C += A.B on
numpy arrays (views with padded rows allowed) -- and raises AssertionError
when the implementation under test disagrees. ``test_oracle.py`` runs them on
the oracle; ``test_oracle_mutants.py`` runs them on deliberately broken copies
of the oracle to show that each plausible mistake is caught.

Sources of truth:
* hand-computed products (tests/golden/hand_products.txt), Sec. 4.1;
* identity, zero and linearity properties of C += A B;
* the transpose identity (A B)^T = B^T A^T;
* closed forms of the modulo-2^32 result for constant operands;
* numpy's exact int64 matrix product reduced to the low 32 bits, and a
  pure-Python big-integer triple loop, as independent implementations.
"""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NP_T = {"i16": np.int16, "i8": np.int8}
RANGE = {"i16": (-32768, 32767), "i8": (-128, 127)}


def wrap32(x):
    """Reduce integers (python ints or int64 arrays) modulo 2^32 to int32."""
    if isinstance(x, np.ndarray):
        return ((x.astype(np.int64) + (1 << 31)) % (1 << 32) - (1 << 31)).astype(np.int32)
    return ((int(x) + (1 << 31)) % (1 << 32)) - (1 << 31)


def load_golden(name: str = "hand_products.txt"):
    """Parse the hand-computed fixture file into a list of dicts."""
    cases = []
    cur = None
    section = None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = {"name": tok[1], "A": [], "B": [], "C0": [], "expect": []}
                section = None
            elif tok[0] == "dtype":
                cur["dtype"] = tok[1]
            elif tok[0] == "dims":
                cur["m"], cur["n"], cur["k"] = map(int, tok[1:4])
            elif tok[0] in ("A", "B", "C0", "expect"):
                section = tok[0]
            elif tok[0] == "end":
                t = NP_T[cur["dtype"]]
                cur["A"] = np.array(cur["A"], dtype=t).reshape(cur["m"], cur["k"])
                cur["B"] = np.array(cur["B"], dtype=t).reshape(cur["k"], cur["n"])
                cur["C0"] = np.array(cur["C0"], dtype=np.int32).reshape(cur["m"], cur["n"])
                cur["expect"] = np.array(cur["expect"], dtype=np.int64).reshape(
                    cur["m"], cur["n"]).astype(np.int32)
                cases.append(cur)
                cur = None
            else:
                cur[section].append([int(v) for v in tok])
    return cases


def numpy_reference(A, B, C0):
    """Exact int64 product via numpy (an independent library routine), then
    the low 32 bits."""
    return wrap32(A.astype(np.int64) @ B.astype(np.int64) + C0.astype(np.int64))


def python_bruteforce(A, B, C0):
    """Pure-Python big-integer triple loop (independent, tiny sizes only)."""
    m, k = A.shape
    n = B.shape[1]
    out = np.empty((m, n), dtype=np.int32)
    for i in range(m):
        for j in range(n):
            s = int(C0[i, j])
            for p in range(k):
                s += int(A[i, p]) * int(B[p, j])
            out[i, j] = wrap32(s)
    return out


def _run(gemm, A, B, C0):
    C = C0.copy()
    gemm(A, B, C)
    return C


def pin_hand_products(gemm):
    for c in load_golden():
        got = _run(gemm, c["A"], c["B"], c["C0"])
        assert np.array_equal(got, c["expect"]), (c["name"], got, c["expect"])


def pin_identity_and_zero(gemm):
    rng = np.random.default_rng(101)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        for (m, k) in ((1, 1), (5, 7), (33, 17)):
            A = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
            C0 = rng.integers(-(1 << 30), 1 << 30, size=(m, k), dtype=np.int32, endpoint=True)
            eye = np.eye(k, dtype=NP_T[dt])
            assert np.array_equal(_run(gemm, A, eye, C0), wrap32(C0.astype(np.int64) + A))
            Z = np.zeros((k, k), dtype=NP_T[dt])
            assert np.array_equal(_run(gemm, A, Z, C0), C0)
            Za = np.zeros((m, m), dtype=NP_T[dt])
            Am = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
            Cm = rng.integers(-5, 5, size=(m, k), dtype=np.int32, endpoint=True)
            assert np.array_equal(_run(gemm, Za, Am, Cm), Cm)
            # I * A = A as well (identity on the left exercises the other operand)
            eyem = np.eye(m, dtype=NP_T[dt])
            assert np.array_equal(_run(gemm, eyem, A, np.zeros_like(C0)),
                                  A.astype(np.int32))


def pin_linearity(gemm):
    """A (B1 + B2) = A B1 + A B2 modulo 2^32, applied as two updates."""
    rng = np.random.default_rng(202)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        m, n, k = 19, 23, 41
        A = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
        B1 = rng.integers(lo // 2, hi // 2, size=(k, n), dtype=NP_T[dt], endpoint=True)
        B2 = rng.integers(lo // 2, hi // 2, size=(k, n), dtype=NP_T[dt], endpoint=True)
        C0 = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n), dtype=np.int32, endpoint=True)
        both = _run(gemm, A, (B1.astype(np.int32) + B2).astype(NP_T[dt]), C0)
        step = _run(gemm, A, B1, C0)
        step = _run(gemm, A, B2, step)
        assert np.array_equal(both, step)


def pin_transpose(gemm):
    """(A B)^T = B^T A^T: the product computed with the roles swapped."""
    rng = np.random.default_rng(303)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        m, n, k = 13, 29, 37
        A = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
        B = rng.integers(lo, hi, size=(k, n), dtype=NP_T[dt], endpoint=True)
        C0 = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n), dtype=np.int32, endpoint=True)
        direct = _run(gemm, A, B, C0)
        swapped = _run(gemm, np.ascontiguousarray(B.T), np.ascontiguousarray(A.T),
                       np.ascontiguousarray(C0.T))
        assert np.array_equal(direct, swapped.T)


def pin_closed_forms(gemm):
    # int16 (-32768)^2 = 2^30: C = k 2^30 mod 2^32 -> 2^30, -2^31, -2^30, 0, ...
    expect_min = {1: 1 << 30, 2: -(1 << 31), 3: -(1 << 30), 4: 0, 5: 1 << 30, 6: -(1 << 31)}
    for k, v in expect_min.items():
        A = np.full((3, k), -32768, np.int16)
        B = np.full((k, 2), -32768, np.int16)
        got = _run(gemm, A, B, np.zeros((3, 2), np.int32))
        assert np.all(got == v), (k, got)
    # int16 32767^2 = 2^30 - 2^16 + 1
    for k in (1, 2, 3, 5, 64, 1000):
        A = np.full((2, k), 32767, np.int16)
        B = np.full((k, 3), 32767, np.int16)
        got = _run(gemm, A, B, np.zeros((2, 3), np.int32))
        assert np.all(got == wrap32(k * ((1 << 30) - (1 << 16) + 1))), k
    # int8 (-128)^2 = 16384, no wraparound below k = 131072
    for k in (1, 7, 300, 4096):
        A = np.full((2, k), -128, np.int8)
        B = np.full((k, 2), -128, np.int8)
        got = _run(gemm, A, B, np.zeros((2, 2), np.int32))
        assert np.all(got == 16384 * k), k
    # A[i,p] = p, B = 1: C[i,j] = k(k-1)/2 for every i, j
    for k in (1, 2, 10, 255, 256, 300):
        A = np.tile(np.arange(k, dtype=np.int16), (4, 1))
        B = np.ones((k, 5), np.int16)
        got = _run(gemm, A, B, np.zeros((4, 5), np.int32))
        assert np.all(got == k * (k - 1) // 2), k
    # A[i,p] = i + 1 (rows differ), B[p,j] = j - 2 (columns differ, signed):
    # C[i,j] = k (i + 1)(j - 2); pins row/column indexing and the sign.
    k = 9
    A = np.repeat(np.arange(1, 5, dtype=np.int8)[:, None], k, axis=1)
    B = np.repeat(np.arange(-2, 4, dtype=np.int8)[None, :], k, axis=0)
    got = _run(gemm, A, B, np.zeros((4, 6), np.int32))
    want = np.array([[k * (i + 1) * (j - 2) for j in range(6)] for i in range(4)], np.int32)
    assert np.array_equal(got, want)


def pin_library_crosscheck(gemm, sizes=None):
    """Random shapes against numpy's exact int64 product (low 32 bits)."""
    rng = np.random.default_rng(404)
    if sizes is None:
        sizes = [(1, 1, 1), (2, 3, 5), (17, 1, 9), (1, 31, 8), (64, 64, 64),
                 (33, 65, 129), (127, 95, 300), (200, 256, 511)]
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        for (m, n, k) in sizes:
            A = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
            B = rng.integers(lo, hi, size=(k, n), dtype=NP_T[dt], endpoint=True)
            C0 = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n), dtype=np.int32,
                              endpoint=True)
            got = _run(gemm, A, B, C0)
            assert np.array_equal(got, numpy_reference(A, B, C0)), (dt, m, n, k)


def pin_bruteforce(gemm):
    """Tiny shapes against a pure-Python big-integer loop."""
    rng = np.random.default_rng(505)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        for (m, n, k) in ((1, 1, 1), (2, 3, 4), (4, 1, 6), (3, 5, 2), (6, 6, 6)):
            A = rng.integers(lo, hi, size=(m, k), dtype=NP_T[dt], endpoint=True)
            B = rng.integers(lo, hi, size=(k, n), dtype=NP_T[dt], endpoint=True)
            C0 = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n), dtype=np.int32,
                              endpoint=True)
            assert np.array_equal(_run(gemm, A, B, C0), python_bruteforce(A, B, C0))


def pin_padding(gemm):
    """Padded leading dimensions: the product uses only the logical windows
    and the padding of C is left untouched."""
    rng = np.random.default_rng(606)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        m, n, k = 7, 9, 11
        Ap = rng.integers(lo, hi, size=(m, k + 5), dtype=NP_T[dt], endpoint=True)
        Bp = rng.integers(lo, hi, size=(k, n + 3), dtype=NP_T[dt], endpoint=True)
        Cp = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n + 4), dtype=np.int32,
                          endpoint=True)
        before = Cp.copy()
        A, B, C = Ap[:, :k], Bp[:, :n], Cp[:, :n]
        want = numpy_reference(np.ascontiguousarray(A), np.ascontiguousarray(B),
                               np.ascontiguousarray(C))
        gemm(A, B, C)
        assert np.array_equal(Cp[:, :n], want)
        assert np.array_equal(Cp[:, n:], before[:, n:])


def pin_degenerate(gemm):
    """k = 0 leaves C unchanged; m = 0 or n = 0 is a no-op."""
    for dt in ("i16", "i8"):
        C0 = np.arange(12, dtype=np.int32).reshape(3, 4) - 6
        A = np.zeros((3, 0), NP_T[dt])
        B = np.zeros((0, 4), NP_T[dt])
        assert np.array_equal(_run(gemm, A, B, C0), C0)
        _run(gemm, np.zeros((0, 5), NP_T[dt]), np.ones((5, 4), NP_T[dt]),
             np.zeros((0, 4), np.int32))
        _run(gemm, np.ones((3, 5), NP_T[dt]), np.ones((5, 0), NP_T[dt]),
             np.zeros((3, 0), np.int32))


ALL_PINS = [pin_hand_products, pin_identity_and_zero, pin_linearity, pin_transpose,
            pin_closed_forms, pin_library_crosscheck, pin_bruteforce, pin_padding,
            pin_degenerate]
