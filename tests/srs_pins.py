"""Pins of the int16-output (shift-round-saturate) oracle: hand-worked cases,
an independent pure-Python implementation, the reduction to the plain GEMM
when nothing saturates or shifts, independence of the block size in that
case, and closed forms of saturation. Each pin takes the function under test
with the signature of ``oracle.igemm_srs`` and raises AssertionError."""
from __future__ import annotations

import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
NP_T = {"i16": np.int16, "i8": np.int8}


def load_golden(name="srs_hand.txt"):
    cases, cur, key = [], None, None
    for raw in open(os.path.join(HERE, "golden", name)):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        parts = line.split()
        tag = parts[0]
        if tag == "case":
            cur = {"name": parts[1]}
        elif tag == "end":
            cases.append(cur)
            cur = None
        elif tag == "dtype":
            cur["dtype"] = parts[1]
        elif tag == "shape":
            cur["shape"] = tuple(int(x) for x in parts[1:])
        elif tag == "srs":
            cur["srs"] = tuple(int(x) for x in parts[1:])
        else:
            cur[tag] = [int(x) for x in parts[1:]]
    return cases


def pin_golden(srs):
    cases = load_golden()
    assert len(cases) >= 10
    for c in cases:
        m, n, k = c["shape"]
        kc, shift, rnd = c["srs"]
        t = NP_T[c["dtype"]]
        A = np.array(c["A"], dtype=t).reshape(m, k)
        B = np.array(c["B"], dtype=t).reshape(k, n)
        C = np.array(c["C0"], dtype=np.int16).reshape(m, n)
        srs(A, B, C, kc, shift, bool(rnd))
        want = np.array(c["expect"], dtype=np.int16).reshape(m, n)
        assert np.array_equal(C, want), f"{c['name']}: got {C.tolist()} want {want.tolist()}"


def python_srs(A, B, C0, kc, shift, rnd):
    """Independent reference: Python integers, floor division by //."""
    m, k = A.shape
    n = B.shape[1]
    blk = k if kc == 0 else kc
    half = (1 << (shift - 1)) if (rnd and shift > 0) else 0
    out = [[int(C0[i, j]) for j in range(n)] for i in range(m)]
    for i in range(m):
        for j in range(n):
            c = out[i][j]
            for p0 in range(0, k, blk):
                acc = sum(int(A[i, p]) * int(B[p, j]) for p in range(p0, min(p0 + blk, k)))
                t = (acc + half) // (1 << shift)
                t = max(-32768, min(32767, t))
                c = (c + t + 32768) % 65536 - 32768
            out[i][j] = c
    return np.array(out, dtype=np.int16).reshape(m, n)


def pin_python_reference(srs):
    rng = np.random.default_rng(71)
    for trial in range(40):
        dt = "i16" if trial % 3 else "i8"
        t = NP_T[dt]
        info = np.iinfo(t)
        m, n, k = (int(x) for x in rng.integers(1, 7, size=3))
        k = int(rng.integers(0, 20))
        # a spread of magnitudes so that some blocks saturate and some do not
        scale = int(rng.choice([3, 60, int(info.max)]))
        A = rng.integers(max(info.min, -scale), min(info.max, scale), size=(m, k), dtype=t,
                         endpoint=True)
        B = rng.integers(info.min, info.max, size=(k, n), dtype=t, endpoint=True)
        C = rng.integers(-32768, 32767, size=(m, n), dtype=np.int16, endpoint=True)
        kc = int(rng.choice([0, 1, 2, 3, 5, 64]))
        shift = int(rng.choice([0, 1, 2, 7, 15, 20, 47]))
        rnd = bool(rng.integers(0, 2))
        want = python_srs(A, B, C, kc, shift, rnd)
        got = srs(A, B, C.copy(), kc, shift, rnd)
        assert np.array_equal(got, want), (trial, kc, shift, rnd)


def pin_reduces_to_gemm(srs):
    """Shift 0, no saturation, no wrap: C0 + A B exactly, for any block size."""
    rng = np.random.default_rng(72)
    for dt in ("i16", "i8"):
        t = NP_T[dt]
        A = rng.integers(-7, 7, size=(9, 20), dtype=t, endpoint=True)
        B = rng.integers(-7, 7, size=(20, 11), dtype=t, endpoint=True)
        C0 = rng.integers(-1000, 1000, size=(9, 11), dtype=np.int16, endpoint=True)
        want = (C0.astype(np.int64) + A.astype(np.int64) @ B.astype(np.int64)).astype(np.int16)
        for kc in (0, 1, 3, 7, 20, 100):
            got = srs(A, B, C0.copy(), kc, 0, False)
            assert np.array_equal(got, want), (dt, kc)
            # rounding does nothing at shift 0
            assert np.array_equal(srs(A, B, C0.copy(), kc, 0, True), want), (dt, kc)


def pin_shift_closed_form(srs):
    """One block, a single product: floor(a*b / 2^s), and +2^(s-1) first with
    rounding, for values of both signs."""
    for a in (-32768, -12345, -5, -1, 1, 5, 12345, 32767):
        for b in (-3, 1, 2, 7):
            for s in (1, 3, 10, 30):
                A = np.array([[a]], dtype=np.int16)
                B = np.array([[b]], dtype=np.int16)
                acc = a * b
                for rnd in (False, True):
                    r = (1 << (s - 1)) if rnd else 0
                    want = max(-32768, min(32767, (acc + r) // (1 << s)))
                    got = int(srs(A, B, np.zeros((1, 1), np.int16), 0, s, rnd)[0, 0])
                    assert got == want, (a, b, s, rnd, got, want)


def pin_saturation_closed_form(srs):
    """All-maximum int16 operands: every block of length L has acc = L*32767^2,
    which saturates to 32767, so C = C0 + nblocks*32767 modulo 2^16; all-
    minimum A with maximum B saturates every block to -32768."""
    for k, kc in ((5, 0), (5, 1), (5, 2), (7, 3), (8, 8), (9, 100)):
        nb = 1 if (kc == 0 or kc >= k) else -(-k // kc)
        A = np.full((2, k), 32767, dtype=np.int16)
        B = np.full((k, 3), 32767, dtype=np.int16)
        C0 = np.array([[0, 1, -1], [32767, -32768, 100]], dtype=np.int16)
        want = ((C0.astype(np.int64) + nb * 32767 + 32768) % 65536 - 32768).astype(np.int16)
        assert np.array_equal(srs(A, B, C0.copy(), kc, 0, False), want), (k, kc)
        An = np.full((2, k), -32768, dtype=np.int16)
        want = ((C0.astype(np.int64) - nb * 32768 + 32768) % 65536 - 32768).astype(np.int16)
        assert np.array_equal(srs(An, B, C0.copy(), kc, 0, False), want), (k, kc)


def pin_block_size_at_least_k(srs):
    """A block size of k or more is one block, as kc = 0."""
    rng = np.random.default_rng(73)
    A = rng.integers(-32768, 32767, size=(4, 13), dtype=np.int16, endpoint=True)
    B = rng.integers(-32768, 32767, size=(13, 5), dtype=np.int16, endpoint=True)
    C0 = rng.integers(-32768, 32767, size=(4, 5), dtype=np.int16, endpoint=True)
    want = srs(A, B, C0.copy(), 0, 9, True)
    for kc in (13, 14, 1000):
        assert np.array_equal(srs(A, B, C0.copy(), kc, 9, True), want), kc


ALL_PINS = [pin_golden, pin_python_reference, pin_reduces_to_gemm, pin_shift_closed_form,
            pin_saturation_closed_form, pin_block_size_at_least_k]
