"""Pins for the CPU convolution oracle: facts fixed by the definition of the
convolution that Sec. 4.2 lowers to one GEMM, and by mathematics, none of
which re-types the oracle's own loop nest.

Each ``pin_*`` function takes ``conv(X, W, Y, stride, pad, dil)`` -- an
in-place Y += conv(X, W) on NHWC / (r, s, c, k) / NHWC numpy arrays -- and
raises AssertionError when the implementation under test disagrees.
``test_conv_oracle.py`` runs them on the oracle and on deliberately broken
copies of it.

Sources of truth:
* hand-computed convolutions (tests/golden/conv_hand.txt);
* an independent numpy formulation: explicit zero padding, then one strided
  slice per filter position and a tensordot over the input channels;
* a delta input, whose output is found by scattering the filter (solving for
  the output positions that read the one non-zero input pixel) rather than by
  gathering;
* the 1x1, stride-1 special case, which is a plain matrix product;
* linearity in X modulo 2^32; output extents of known layers.
"""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
NP_T = {"i16": np.int16, "i8": np.int8}
RANGE = {"i16": (-32768, 32767), "i8": (-128, 127)}


def wrap32(x):
    return ((np.asarray(x, dtype=np.int64) + (1 << 31)) % (1 << 32) - (1 << 31)).astype(np.int32)


def out_dim(size, f, stride, pad, dil):
    span = size + 2 * pad - dil * (f - 1) - 1
    return 0 if span < 0 else span // stride + 1


def load_golden(name="conv_hand.txt"):
    cases, cur = [], None
    for raw in open(os.path.join(GOLDEN, name)):
        line = raw.strip()
        if not line or line.startswith("#"):
            continue
        key, *rest = line.split()
        if key == "case":
            cur = {"name": rest[0]}
        elif key == "end":
            cases.append(cur)
            cur = None
        elif key in ("dtype",):
            cur[key] = rest[0]
        else:
            cur[key] = [int(v) for v in rest]
    return cases


def numpy_conv(X, W, stride, pad, dil):
    """Exact convolution in int64 by padding and strided slicing."""
    n, h, w, c = X.shape
    r, s, _, k = W.shape
    oh = out_dim(h, r, stride[0], pad[0], dil[0])
    ow = out_dim(w, s, stride[1], pad[1], dil[1])
    Xp = np.pad(X.astype(np.int64), ((0, 0), (pad[0], pad[0]), (pad[1], pad[1]), (0, 0)))
    out = np.zeros((n, oh, ow, k), dtype=np.int64)
    if oh == 0 or ow == 0:
        return out
    for fy in range(r):
        for fx in range(s):
            y0, x0 = fy * dil[0], fx * dil[1]
            patch = Xp[:, y0:y0 + stride[0] * (oh - 1) + 1:stride[0],
                       x0:x0 + stride[1] * (ow - 1) + 1:stride[1], :]
            out += np.tensordot(patch, W[fy, fx].astype(np.int64), axes=([3], [0]))
    return out


def _run(conv, X, W, Y0, stride, pad, dil):
    Y = Y0.copy()
    conv(X, W, Y, stride, pad, dil)
    return Y


def pin_golden(conv):
    cases = load_golden()
    assert len(cases) >= 8
    for cs in cases:
        t = NP_T[cs["dtype"]]
        n, h, w, c, k, r, s = cs["shape"]
        sh, sw, ph, pw, dh, dw = cs["conv"]
        oh, ow = out_dim(h, r, sh, ph, dh), out_dim(w, s, sw, pw, dw)
        X = np.array(cs["X"], dtype=t).reshape(n, h, w, c)
        W = np.array(cs["W"], dtype=t).reshape(r, s, c, k)
        Y0 = np.array(cs["Y0"], dtype=np.int32).reshape(n, oh, ow, k)
        want = np.array(cs["expect"], dtype=np.int64).reshape(n, oh, ow, k)
        got = _run(conv, X, W, Y0, (sh, sw), (ph, pw), (dh, dw))
        assert np.array_equal(got, wrap32(want)), (cs["name"], got.ravel(), want.ravel())


def _random_case(rng, dt):
    lo, hi = RANGE[dt]
    n = int(rng.integers(1, 3))
    h, w = (int(v) for v in rng.integers(1, 8, 2))
    c, k = int(rng.integers(1, 6)), int(rng.integers(1, 5))
    r, s = (int(v) for v in rng.integers(1, 4, 2))
    stride = tuple(int(v) for v in rng.integers(1, 4, 2))
    pad = tuple(int(v) for v in rng.integers(0, 3, 2))
    dil = tuple(int(v) for v in rng.integers(1, 3, 2))
    X = rng.integers(lo, hi, (n, h, w, c), dtype=NP_T[dt], endpoint=True)
    W = rng.integers(lo, hi, (r, s, c, k), dtype=NP_T[dt], endpoint=True)
    oh, ow = out_dim(h, r, stride[0], pad[0], dil[0]), out_dim(w, s, stride[1], pad[1], dil[1])
    Y0 = rng.integers(-(1 << 31), (1 << 31) - 1, (n, oh, ow, k), dtype=np.int32, endpoint=True)
    return X, W, Y0, stride, pad, dil


def pin_numpy_reference(conv):
    rng = np.random.default_rng(77)
    for i in range(60):
        dt = "i16" if i % 3 else "i8"
        X, W, Y0, stride, pad, dil = _random_case(rng, dt)
        got = _run(conv, X, W, Y0, stride, pad, dil)
        want = wrap32(Y0.astype(np.int64) + numpy_conv(X, W, stride, pad, dil))
        assert np.array_equal(got, want), (i, X.shape, W.shape, stride, pad, dil)


def pin_delta_scatter(conv):
    rng = np.random.default_rng(78)
    for i in range(40):
        n, h, w, c, k = 2, 6, 7, 3, 2
        r, s = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        stride = tuple(int(v) for v in rng.integers(1, 3, 2))
        pad = tuple(int(v) for v in rng.integers(0, 3, 2))
        dil = tuple(int(v) for v in rng.integers(1, 3, 2))
        oh, ow = out_dim(h, r, stride[0], pad[0], dil[0]), out_dim(w, s, stride[1], pad[1], dil[1])
        b, y, x, ci = (int(rng.integers(0, v)) for v in (n, h, w, c))
        v = int(rng.integers(-300, 301))
        X = np.zeros((n, h, w, c), np.int16)
        X[b, y, x, ci] = v
        W = rng.integers(-1000, 1000, (r, s, c, k), dtype=np.int16, endpoint=True)
        want = np.zeros((n, oh, ow, k), np.int64)
        # The input pixel (y, x) is read by output (oy, ox) through filter
        # position (fy, fx) exactly when oy*sh - ph + fy*dh == y (and alike in x).
        for fy in range(r):
            ty = y + pad[0] - fy * dil[0]
            if ty % stride[0] or not 0 <= ty // stride[0] < oh:
                continue
            for fx in range(s):
                tx = x + pad[1] - fx * dil[1]
                if tx % stride[1] or not 0 <= tx // stride[1] < ow:
                    continue
                want[b, ty // stride[0], tx // stride[1]] += v * W[fy, fx, ci].astype(np.int64)
        got = _run(conv, X, W, np.zeros((n, oh, ow, k), np.int32), stride, pad, dil)
        assert np.array_equal(got, wrap32(want)), (i, r, s, stride, pad, dil, (b, y, x, ci))


def pin_one_by_one_is_matmul(conv):
    rng = np.random.default_rng(79)
    for dt in ("i16", "i8"):
        lo, hi = RANGE[dt]
        n, h, w, c, k = 2, 5, 3, 7, 6
        X = rng.integers(lo, hi, (n, h, w, c), dtype=NP_T[dt], endpoint=True)
        W = rng.integers(lo, hi, (1, 1, c, k), dtype=NP_T[dt], endpoint=True)
        Y0 = rng.integers(-1000, 1000, (n, h, w, k), dtype=np.int32, endpoint=True)
        got = _run(conv, X, W, Y0, (1, 1), (0, 0), (1, 1))
        prod = X.reshape(-1, c).astype(np.int64) @ W.reshape(c, k).astype(np.int64)
        want = wrap32(Y0.reshape(-1, k).astype(np.int64) + prod).reshape(n, h, w, k)
        assert np.array_equal(got, want), dt


def pin_linearity(conv):
    rng = np.random.default_rng(80)
    X1 = rng.integers(-16384, 16383, (1, 6, 5, 4), dtype=np.int16, endpoint=True)
    X2 = rng.integers(-16384, 16383, (1, 6, 5, 4), dtype=np.int16, endpoint=True)
    W = rng.integers(-32768, 32767, (3, 2, 4, 3), dtype=np.int16, endpoint=True)
    args = ((2, 1), (1, 1), (1, 2))
    oh, ow = out_dim(6, 3, 2, 1, 1), out_dim(5, 2, 1, 1, 2)
    Z = np.zeros((1, oh, ow, 3), np.int32)
    y12 = _run(conv, (X1 + X2).astype(np.int16), W, Z, *args)
    y1 = _run(conv, X1, W, Z, *args)
    y2 = _run(conv, X2, W, Z, *args)
    assert np.array_equal(y12, wrap32(y1.astype(np.int64) + y2))


def pin_out_dims(conv):
    # ResNet-50 layers at 224 x 224: 7x7/2 pad 3 -> 112; 3x3/2 pad 1 on 56 -> 28;
    # 1x1 on 56 -> 56; a window larger than the padded input gives no output.
    assert out_dim(224, 7, 2, 3, 1) == 112
    assert out_dim(56, 3, 2, 1, 1) == 28
    assert out_dim(56, 1, 1, 0, 1) == 56
    assert out_dim(2, 5, 1, 1, 1) == 0
    X = np.ones((1, 2, 2, 1), np.int16)
    W = np.ones((5, 5, 1, 1), np.int16)
    Y = np.zeros((1, 0, 0, 1), np.int32)
    conv(X, W, Y, (1, 1), (1, 1), (1, 1))  # nothing to compute, and no error


ALL_PINS = [pin_golden, pin_numpy_reference, pin_delta_scatter, pin_one_by_one_is_matmul,
            pin_linearity, pin_out_dims]
