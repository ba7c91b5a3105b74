"""The CPU convolution oracle against its pins, and plausible mistakes planted
in copies of it (on the CPU), each of which some pin must catch."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import conv_pins as pins
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "igemm_oracle.c")


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_conv_pin(pin):
    pin(oracle.conv2d)


def test_oracle_conv_out_dim_matches_pin_formula():
    for args in ((224, 7, 2, 3, 1), (56, 3, 2, 1, 1), (9, 3, 1, 0, 4), (3, 5, 1, 0, 1)):
        assert oracle.conv2d_out_dim(*args) == pins.out_dim(*args)
    assert oracle.conv2d_out_dim(5, 0, 1, 0, 1) == -1


MUTANTS = [
    ("filter_rows_for_cols", "const T *wp = W + (fy * s + fx) * c * k;",
     "const T *wp = W + (fx * r + fy) * c * k;"),
    ("no_dilation", "const int64_t iy = oy * stride_h - pad_h + fy * dil_h;",
     "const int64_t iy = oy * stride_h - pad_h + fy;"),
    ("stride_on_filter", "const int64_t ix = ox * stride_w - pad_w + fx * dil_w;",
     "const int64_t ix = ox - pad_w + fx * stride_w;"),
    ("pad_sign", "const int64_t iy = oy * stride_h - pad_h + fy * dil_h;",
     "const int64_t iy = oy * stride_h + pad_h + fy * dil_h;"),
    ("dropped_Y0", "acc[co] = (int64_t)y[co];", "acc[co] = 0;"),
    ("channel_stride_in_W", "const T *wrow = wp + ci * k;", "const T *wrow = wp + ci;"),
    ("first_channel_only", "const int64_t xv = (int64_t)xp[ci];",
     "const int64_t xv = (int64_t)xp[0];"),
    ("out_dim_ceil", "return span < 0 ? 0 : span / stride + 1;",
     "return span < 0 ? 0 : (span + stride - 1) / stride + 1;"),
]


def _conv_from(tmp_path, name, find, repl):
    text = open(SRC).read()
    assert find in text, name
    src = tmp_path / f"{name}.c"
    src.write_text(text.replace(find, repl))
    lib_path = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fopenmp", "-fPIC", "-shared", str(src), "-o",
                    str(lib_path)], check=True)
    lib = ctypes.CDLL(str(lib_path))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    for nm in ("oracle_conv2d_i16", "oracle_conv2d_i8"):
        getattr(lib, nm).argtypes = [i64] * 13 + [vp, vp, vp]
        getattr(lib, nm).restype = ctypes.c_int
    lib.oracle_conv2d_out_dim.argtypes = [i64] * 5
    lib.oracle_conv2d_out_dim.restype = i64

    def conv(X, W, Y, stride, pad, dil):
        n, h, w, c = X.shape
        r, s, _, k = W.shape
        oh = lib.oracle_conv2d_out_dim(h, r, stride[0], pad[0], dil[0])
        ow = lib.oracle_conv2d_out_dim(w, s, stride[1], pad[1], dil[1])
        if Y.shape != (n, oh, ow, k):
            raise AssertionError(f"output extent {(oh, ow)} for Y {Y.shape}")
        fn = lib.oracle_conv2d_i16 if X.dtype == np.int16 else lib.oracle_conv2d_i8
        st = fn(n, h, w, c, k, r, s, stride[0], stride[1], pad[0], pad[1], dil[0], dil[1],
                X.ctypes.data_as(vp), W.ctypes.data_as(vp), Y.ctypes.data_as(vp))
        if st != 0:
            raise AssertionError(f"status {st}")
        return Y
    return conv


@pytest.mark.parametrize("mut", MUTANTS, ids=lambda m: m[0])
def test_conv_pins_catch_mutant(tmp_path, mut):
    conv = _conv_from(tmp_path, *mut)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(conv)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {mut[0]} passed every pin"


def test_unmodified_conv_copy_passes_every_pin(tmp_path):
    conv = _conv_from(tmp_path, "unmodified", "static int32_t wrap_to_i32",
                      "static int32_t wrap_to_i32")
    for pin in pins.ALL_PINS:
        pin(conv)
