"""Seeded synthetic inputs for integer GEMM C += A.B.

This module only draws numbers. It holds none of the GEMM arithmetic, so the
CPU oracle (under ``oracle/``) and the GPU path can both take their inputs
from here without sharing any of the method.

Workloads (all row-major, C is int32):

* ``i16_256``      int16 m=n=k=256, A,B uniform over the full int16 range,
                   C zero, seed 0.
* ``i16_4096``     int16 m=n=k=4096, A,B uniform over the full range,
                   C uniform in [-2^20, 2^20], seed 1.
* ``i8_8192``      int8 m=n=k=8192, A,B uniform in [-128,127], C zero, seed 2.
* ``i16_conv``     six int16 GEMMs shaped like the im2row lowering of the
                   convolutions of a 50-layer residual CNN at batch 1 on a
                   224x224 input (m = output pixels, n = output channels,
                   k = input channels x kernel window; the lowering of a
                   convolution to one GEMM is Sec. 4.2). A uniform in [0,255]
                   (activations), B = rint(normal(0,32)) clipped to int16
                   (weights), C zero; layer i uses seed 40+i.
* ``CONV2D_CASES`` the six ``i16_conv`` layers as real convolutions from an
                   NHWC image (implicit GEMM), seeds 60+i; ``CONV2D_B32_CASES``
                   the same at batch 32, seeds 70+i.
* ``i16_paper``    the paper's GEMM shape (4096, 4096, 290), int16 with the
                   recipe of i16_4096, seed 3 (context, not a graded workload).
* ``i8_skinny``    six int8 GEMMs shaped like the projections of a 7B-class
                   decoder at small batch (one large dimension and two small
                   ones, Sec. 2 and Sec. 4.2): m in {1,8,32} with (n,k) in
                   {(4096,4096), (11008,4096)}; A uniform in [-128,127],
                   B = rint(normal(0,20)) clipped to [-128,127], C zero;
                   shape i uses seed 50+i.
* ``i16_skinny``   the ``i8_skinny`` shapes in int16 (context, not a graded
                   workload): A uniform in [-32768,32767], B =
                   rint(normal(0,5120)) clipped to int16, C zero; shape i uses
                   seed 80+i.

Conventions: numpy ``default_rng(seed)`` (PCG64); draws in the order A, B, C;
uniform integer ranges include both ends; "normal clipped" rounds with
``rint`` (ties to even) and then clips. No dataset, image or trained weight
is involved: every tensor is i.i.d. synthetic with the stated distribution.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

I16_MIN, I16_MAX = -32768, 32767
I8_MIN, I8_MAX = -128, 127


@dataclass(frozen=True)
class Dist:
    """A value distribution for one operand."""

    kind: str  # "uniform" | "normal_clip" | "zero"
    lo: int = 0
    hi: int = 0
    sigma: float = 0.0


@dataclass(frozen=True)
class Case:
    """One GEMM problem: shape, operand type and value distributions."""

    name: str
    dtype: str  # "i16" | "i8"
    m: int
    n: int
    k: int
    a: Dist
    b: Dist
    c: Dist
    seed: int


@dataclass(frozen=True)
class Workload:
    name: str
    cases: Tuple[Case, ...]
    description: str = ""


def _np_dtype(dtype: str):
    if dtype == "i16":
        return np.int16
    if dtype == "i8":
        return np.int8
    raise ValueError(f"unknown operand dtype {dtype!r}")


def draw(rng: np.random.Generator, dist: Dist, shape, dtype) -> np.ndarray:
    """Draw one operand. ``dtype`` is the numpy storage type."""
    if dist.kind == "zero":
        return np.zeros(shape, dtype=dtype)
    if dist.kind == "uniform":
        return rng.integers(dist.lo, dist.hi, size=shape, dtype=dtype, endpoint=True)
    if dist.kind == "normal_clip":
        x = np.rint(rng.normal(0.0, dist.sigma, size=shape))
        return np.clip(x, dist.lo, dist.hi).astype(dtype)
    raise ValueError(f"unknown distribution {dist.kind!r}")


def generate(case: Case, seed: Optional[int] = None):
    """Return (A, B, C0) as C-contiguous numpy arrays for ``case``.

    A is m x k and B is k x n in the case's operand type; C0 is m x n int32.
    """
    rng = np.random.default_rng(case.seed if seed is None else seed)
    et = _np_dtype(case.dtype)
    A = draw(rng, case.a, (case.m, case.k), et)
    B = draw(rng, case.b, (case.k, case.n), et)
    C = draw(rng, case.c, (case.m, case.n), np.int32)
    return A, B, C


def random_operands(dtype: str, m: int, n: int, k: int, seed: int,
                    c_range: int = 1 << 20, lda: Optional[int] = None,
                    ldb: Optional[int] = None, ldc: Optional[int] = None):
    """Full-range random operands with optional padded leading dimensions.

    Returns (A, B, C) where each is a 2-D array whose row length is the
    leading dimension (>= the logical width); padding is filled with values
    from the same distribution so an out-of-bounds read changes the result
    and an out-of-bounds write is visible.
    """
    et = _np_dtype(dtype)
    lo, hi = (I16_MIN, I16_MAX) if dtype == "i16" else (I8_MIN, I8_MAX)
    lda = k if lda is None else lda
    ldb = n if ldb is None else ldb
    ldc = n if ldc is None else ldc
    rng = np.random.default_rng(seed)
    A = rng.integers(lo, hi, size=(m, max(lda, 1)), dtype=et, endpoint=True)
    B = rng.integers(lo, hi, size=(k, max(ldb, 1)), dtype=et, endpoint=True)
    C = rng.integers(-c_range, c_range, size=(m, max(ldc, 1)), dtype=np.int32,
                     endpoint=True)
    return A, B, C


def random_conv_operands(dtype: str, n: int, h: int, w: int, c: int, k: int, r: int, s: int,
                         oh: int, ow: int, seed: int, y_range: int = 1 << 20):
    """Full-range random X (n x h x w x c), W (r x s x c x k) and a random
    starting Y (n x oh x ow x k int32) for a convolution, drawn in that
    order."""
    et = _np_dtype(dtype)
    lo, hi = (I16_MIN, I16_MAX) if dtype == "i16" else (I8_MIN, I8_MAX)
    rng = np.random.default_rng(seed)
    X = rng.integers(lo, hi, size=(n, h, w, c), dtype=et, endpoint=True)
    W = rng.integers(lo, hi, size=(r, s, c, k), dtype=et, endpoint=True)
    Y = rng.integers(-y_range, y_range, size=(n, oh, ow, k), dtype=np.int32, endpoint=True)
    return X, W, Y


_U16 = Dist("uniform", I16_MIN, I16_MAX)
_U8 = Dist("uniform", I8_MIN, I8_MAX)
_ZERO = Dist("zero")

CONV_SHAPES = (
    (12544, 64, 147),
    (3136, 64, 576),
    (3136, 256, 64),
    (784, 128, 1152),
    (196, 256, 2304),
    (49, 512, 4608),
)

SKINNY_SHAPES = (
    (1, 4096, 4096),
    (8, 4096, 4096),
    (32, 4096, 4096),
    (1, 11008, 4096),
    (8, 11008, 4096),
    (32, 11008, 4096),
)

WORKLOADS = {
    "i16_256": Workload(
        "i16_256",
        (Case("i16_256", "i16", 256, 256, 256, _U16, _U16, _ZERO, 0),),
        "int16 C+=A.B, m=n=k=256, full-range operands, C zero",
    ),
    "i16_4096": Workload(
        "i16_4096",
        (Case("i16_4096", "i16", 4096, 4096, 4096, _U16, _U16,
              Dist("uniform", -(1 << 20), 1 << 20), 1),),
        "int16 C+=A.B, m=n=k=4096, full-range operands, C uniform in +-2^20",
    ),
    "i8_8192": Workload(
        "i8_8192",
        (Case("i8_8192", "i8", 8192, 8192, 8192, _U8, _U8, _ZERO, 2),),
        "int8 C+=A.B, m=n=k=8192, full-range operands, C zero",
    ),
    "i16_conv": Workload(
        "i16_conv",
        tuple(
            Case(f"i16_conv_{i}_{m}x{n}x{k}", "i16", m, n, k,
                 Dist("uniform", 0, 255),
                 Dist("normal_clip", I16_MIN, I16_MAX, 32.0), _ZERO, 40 + i)
            for i, (m, n, k) in enumerate(CONV_SHAPES)
        ),
        "int16 GEMMs shaped like a 50-layer residual CNN's im2row convolutions",
    ),
    "i8_skinny": Workload(
        "i8_skinny",
        tuple(
            Case(f"i8_skinny_{i}_{m}x{n}x{k}", "i8", m, n, k, _U8,
                 Dist("normal_clip", I8_MIN, I8_MAX, 20.0), _ZERO, 50 + i)
            for i, (m, n, k) in enumerate(SKINNY_SHAPES)
        ),
        "int8 skinny GEMMs shaped like 7B-class decoder projections",
    ),
}

# The paper's own GEMM shape (its m_c sweep runs (m, n, k) = (4096, 4096, 290) with
# n_c = n and k_c = k, Sec. 6.4), with the int16 recipe of i16_4096. Context only: it
# is measured and checked like the others but is not one of the graded workloads.
WORKLOADS["i16_paper"] = Workload(
    "i16_paper",
    (Case("i16_paper_4096x4096x290", "i16", 4096, 4096, 290, _U16, _U16,
          Dist("uniform", -(1 << 20), 1 << 20), 3),),
    "int16 C+=A.B, (m, n, k) = (4096, 4096, 290), full-range operands, C uniform in +-2^20",
)

# The same projection shapes with int16 operands (context only, like i16_paper).
WORKLOADS["i16_skinny"] = Workload(
    "i16_skinny",
    tuple(
        Case(f"i16_skinny_{i}_{m}x{n}x{k}", "i16", m, n, k, _U16,
             Dist("normal_clip", I16_MIN, I16_MAX, 5120.0), _ZERO, 80 + i)
        for i, (m, n, k) in enumerate(SKINNY_SHAPES)
    ),
    "int16 skinny GEMMs shaped like 7B-class decoder projections",
)

ORDER: List[str] = ["i16_256", "i16_4096", "i8_8192", "i16_conv", "i8_skinny"]


@dataclass(frozen=True)
class ConvCase:
    """One convolution Y += conv(X, W): X n x h x w x c (NHWC), W r x s x c x k,
    Y n x oh x ow x k, with strides, zero padding and dilations."""

    name: str
    dtype: str
    n: int
    h: int
    w: int
    c: int
    k: int
    r: int
    s: int
    stride: Tuple[int, int]
    pad: Tuple[int, int]
    dil: Tuple[int, int]
    x: Dist
    wt: Dist
    seed: int

    def out_hw(self):
        def od(size, f, st, pd, dl):
            span = size + 2 * pd - dl * (f - 1) - 1
            return 0 if span < 0 else span // st + 1
        return (od(self.h, self.r, self.stride[0], self.pad[0], self.dil[0]),
                od(self.w, self.s, self.stride[1], self.pad[1], self.dil[1]))

    def gemm_shape(self):
        """(m, n, k) of the GEMM that IM2ROW lowers this convolution to."""
        oh, ow = self.out_hw()
        return self.n * oh * ow, self.k, self.r * self.s * self.c


def generate_conv(case: ConvCase, seed: Optional[int] = None):
    """Return (X, W, Y0) for ``case``: draws in the order X, W; Y0 is zero."""
    rng = np.random.default_rng(case.seed if seed is None else seed)
    et = _np_dtype(case.dtype)
    X = draw(rng, case.x, (case.n, case.h, case.w, case.c), et)
    W = draw(rng, case.wt, (case.r, case.s, case.c, case.k), et)
    oh, ow = case.out_hw()
    Y = np.zeros((case.n, oh, ow, case.k), dtype=np.int32)
    return X, W, Y


# The six layers of the conv-shaped GEMM set as convolutions on an NHWC image
# (batch 1, 224 x 224 input): the 7x7 stride-2 stem, a 3x3 and a 1x1 layer at
# 56 x 56, and the 3x3 stride-2 layers that open the next three stages. Their
# IM2ROW lowerings have exactly the GEMM shapes of ``i16_conv``. Activations
# uniform in [0, 255], weights rint(normal(0, 32)) clipped; layer i uses seed
# 60 + i.
CONV2D_LAYERS = (
    ("stem_7x7s2", 224, 3, 64, 7, 2, 3),
    ("c2_3x3", 56, 64, 64, 3, 1, 1),
    ("c2_1x1", 56, 64, 256, 1, 1, 0),
    ("c3_3x3s2", 56, 128, 128, 3, 2, 1),
    ("c4_3x3s2", 28, 256, 256, 3, 2, 1),
    ("c5_3x3s2", 14, 512, 512, 3, 2, 1),
)
CONV2D_CASES = tuple(
    ConvCase(f"i16_conv2d_{i}_{nm}", "i16", 1, hw, hw, c, k, f, f, (st, st), (pd, pd), (1, 1),
             Dist("uniform", 0, 255), Dist("normal_clip", I16_MIN, I16_MAX, 32.0), 60 + i)
    for i, (nm, hw, c, k, f, st, pd) in enumerate(CONV2D_LAYERS)
)
# The same layers at batch 32, where the output traffic rather than the
# launch latency bounds each layer; seeds 70 + i.
CONV2D_B32_CASES = tuple(
    ConvCase(f"i16_conv2d_b32_{i}_{nm}", "i16", 32, hw, hw, c, k, f, f, (st, st), (pd, pd),
             (1, 1), Dist("uniform", 0, 255), Dist("normal_clip", I16_MIN, I16_MAX, 32.0), 70 + i)
    for i, (nm, hw, c, k, f, st, pd) in enumerate(CONV2D_LAYERS)
)


def ops(case: Case) -> int:
    """Arithmetic operations of one GEMM, counting a multiply-add as two."""
    return 2 * case.m * case.n * case.k


def algorithmic_bytes(case: Case) -> int:
    """A and B read once, C read and written once as int32."""
    e = 2 if case.dtype == "i16" else 1
    return case.m * case.k * e + case.k * case.n * e + 8 * case.m * case.n
