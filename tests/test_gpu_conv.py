"""GPU parity of the convolution entry points (IM2ROW lowering gathered while
the A tiles are staged) against the oracle's direct convolution, element by
element and bit-exact, through the C ABI."""
import numpy as np
import pytest

import workloads
from gpu_util import to_device

pytestmark = pytest.mark.gpu

CONV_KERNELS = {"i16": ("i16_128x128", "i16_64x64", "i16_32x128", "i16_16x128"),
                "i8": ("i8_32x256", "i8_16x256")}
SENTINEL = 0x5A5A5A5A


def _ig():
    import paper_2302_07594_amd as ig
    return ig


def _kid(name):
    ig = _ig()
    return [ig.igemm_kernel_name(i) for i in range(ig.igemm_num_kernels())].index(name)


def _oracle(X, W, Y, stride, pad, dil):
    import oracle
    out = Y.copy()
    oracle.conv2d(X, W, out, stride, pad, dil)
    return out


def _gpu(X, W, Y, stride, pad, dil, kernel=-1, split=-1, x_off=0, w_off=0):
    """Run Y += conv(X, W) through igemm_conv2d_ex; Y sits in a larger buffer
    whose tail holds sentinels that must survive. Returns Y as numpy."""
    import torch
    ig = _ig()
    n, h, w, c = X.shape
    r, s, _, k = W.shape
    Xd = to_device(X, x_off)
    Wd = to_device(W, w_off)
    flat = torch.full((Y.size + 64,), SENTINEL, dtype=torch.int32, device="cuda")
    flat[:Y.size].copy_(torch.from_numpy(Y.reshape(-1)).cuda())
    es = 2 if X.dtype == np.int16 else 1
    d = ig.conv_desc(n, h, w, c, k, r, s, stride, pad, dil)
    st = ig.igemm_conv2d_ex(es, d, Xd.data_ptr(), Wd.data_ptr(), flat.data_ptr(),
                            torch.cuda.current_stream().cuda_stream, kernel, split)
    torch.cuda.synchronize()
    assert st == 0, f"status {st}: {ig.igemm_strerror(st)}"
    out = flat.cpu().numpy()
    assert np.all(out[Y.size:] == SENTINEL), "write past the end of Y"
    return out[:Y.size].reshape(Y.shape)


def _describe(got, want, limit=5):
    bad = np.argwhere(got != want)
    lines = [f"{len(bad)} of {got.size} elements differ"]
    for idx in bad[:limit]:
        t = tuple(int(i) for i in idx)
        lines.append(f"  Y{t} got {got[t]} want {want[t]}")
    return "\n".join(lines)


def _check(dt, n, h, w, c, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1), seed=0, **kw):
    ig = _ig()
    oh = ig.igemm_conv2d_out_dim(h, r, stride[0], pad[0], dil[0])
    ow = ig.igemm_conv2d_out_dim(w, s, stride[1], pad[1], dil[1])
    X, W, Y = workloads.random_conv_operands(dt, n, h, w, c, k, r, s, oh, ow, seed)
    want = _oracle(X, W, Y, stride, pad, dil)
    got = _gpu(X, W, Y, stride, pad, dil, **kw)
    assert np.array_equal(got, want), _describe(got, want)
    return got


@pytest.mark.parametrize("case", workloads.CONV2D_CASES, ids=lambda c: c.name)
def test_resnet_layers_full(case):
    """The six network layers at full size with their value distributions
    (automatic plan), every output compared."""
    X, W, Y = workloads.generate_conv(case)
    want = _oracle(X, W, Y, case.stride, case.pad, case.dil)
    got = _gpu(X, W, Y, case.stride, case.pad, case.dil)
    assert np.array_equal(got, want), _describe(got, want)
    assert np.any(got != 0)


@pytest.mark.parametrize("case", workloads.CONV2D_B32_CASES, ids=lambda c: c.name)
def test_resnet_layers_batch32_sampled_images(case):
    """The six layers at batch 32 in the launch configuration the benchmark
    times; images 0, 17 and 31 compared in full with the oracle run on those
    images alone (each output image depends on its own input image only)."""
    X, W, Y = workloads.generate_conv(case)
    got = _gpu(X, W, Y, case.stride, case.pad, case.dil)
    for b in (0, 17, 31):
        want = _oracle(np.ascontiguousarray(X[b:b + 1]), W, np.ascontiguousarray(Y[b:b + 1]),
                       case.stride, case.pad, case.dil)
        assert np.array_equal(got[b:b + 1], want), f"image {b}: " + _describe(got[b:b + 1], want)


# (n, h, w, c, k, r, s, stride, pad, dil): channel counts that take the 16-byte
# gather and ones that do not, windows that straddle image and batch borders,
# strides, dilations, padding wider than the filter, one-pixel outputs.
SHAPES = [
    (1, 9, 11, 8, 40, 3, 3, (1, 1), (1, 1), (1, 1)),
    (2, 13, 10, 16, 70, 3, 3, (2, 2), (1, 1), (1, 1)),
    (3, 7, 7, 3, 33, 7, 7, (2, 2), (3, 3), (1, 1)),
    (1, 12, 17, 5, 129, 3, 2, (1, 2), (2, 0), (2, 1)),
    (2, 6, 6, 32, 17, 1, 1, (1, 1), (0, 0), (1, 1)),
    (1, 10, 9, 24, 64, 5, 3, (3, 1), (4, 2), (1, 3)),
    (4, 5, 5, 1, 7, 2, 2, (1, 1), (0, 0), (1, 1)),
    (1, 3, 3, 64, 256, 3, 3, (1, 1), (1, 1), (1, 1)),
    (2, 4, 4, 48, 9, 4, 4, (1, 1), (0, 0), (1, 1)),   # one output pixel per image
    (1, 20, 3, 72, 300, 3, 1, (2, 1), (0, 5), (1, 1)),  # padding beyond the filter
]


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda t: "x".join(map(str, t[:7])))
def test_every_conv_kernel(dt, shape):
    """Every conv kernel of the type, automatic and forced k slices, on
    ragged shapes (output pixels and channels not multiples of the tile,
    k = r*s*c not a multiple of 64)."""
    n, h, w, c, k, r, s, stride, pad, dil = shape
    seed = 500 + sum(shape[:7])
    for name in CONV_KERNELS[dt]:
        for split in (-1, 1, 3):
            _check(dt, n, h, w, c, k, r, s, stride, pad, dil, seed=seed, kernel=_kid(name),
                   split=split)


# Shapes for the small-output int16 kernel's gather (channels a multiple of
# 64: each k-tile is 64 channels of one filter tap; output channels a
# multiple of 8): padding beyond the filter, strides, dilations, several
# images, taps of several k-tiles, one output pixel per image.
SMALL_SHAPES = [
    (1, 9, 11, 64, 40, 3, 3, (1, 1), (1, 1), (1, 1)),
    (2, 13, 10, 64, 72, 3, 3, (2, 2), (1, 1), (1, 1)),
    (1, 12, 17, 128, 136, 3, 2, (1, 2), (2, 0), (2, 1)),
    (2, 6, 6, 64, 16, 1, 1, (1, 1), (0, 0), (1, 1)),
    (1, 10, 9, 64, 64, 5, 3, (3, 1), (4, 2), (1, 3)),
    (2, 4, 4, 192, 8, 4, 4, (1, 1), (0, 0), (1, 1)),
    (1, 20, 3, 64, 304, 3, 1, (2, 1), (0, 5), (1, 1)),
    (3, 7, 7, 128, 24, 3, 3, (1, 1), (1, 1), (1, 1)),
]


@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=lambda t: "x".join(map(str, t[:7])))
def test_small_kernel_gather(shape):
    """The small-output kernel with A gathered from X (taps outside the image
    read as zeros through the buffer resource), automatic and forced k
    slices, including a short last slice."""
    n, h, w, c, k, r, s, stride, pad, dil = shape
    for split in (-1, 1, 3, 100):
        _check("i16", n, h, w, c, k, r, s, stride, pad, dil, seed=900 + sum(shape[:7]),
               kernel=_kid("i16_small_64x64"), split=split)


RUN_SHAPES = [
    # (n, h, w, c, k, r, s, stride, pad, dil, x_off)
    (1, 224, 224, 3, 64, 7, 7, (2, 2), (3, 3), (1, 1), 0),   # the stem layer
    (2, 17, 13, 3, 16, 7, 7, (2, 2), (3, 3), (1, 1), 1),
    (1, 9, 11, 5, 24, 3, 3, (1, 1), (1, 1), (2, 1), 3),
    (1, 12, 12, 1, 8, 7, 7, (1, 1), (3, 3), (1, 1), 0),      # s c = 7: two runs per chunk
    (1, 10, 10, 100, 16, 3, 3, (1, 1), (1, 1), (1, 1), 1),
    (3, 8, 8, 17, 40, 2, 5, (1, 2), (0, 2), (1, 1), 0),
    (1, 6, 6, 48, 64, 3, 3, (1, 1), (1, 1), (1, 1), 0),
    (1, 20, 20, 64, 64, 3, 3, (1, 1), (1, 1), (1, 1), 1),    # 64 channels, misaligned X
    (1, 9, 9, 8, 16, 3, 1, (1, 1), (1, 0), (2, 3), 0),       # one-column filter, any dilation
]


@pytest.mark.parametrize("shape", RUN_SHAPES, ids=lambda t: "x".join(map(str, t[:7])))
def test_small_kernel_runs(shape):
    """The small-output kernel gathering IM2ROW rows as input runs (any
    channel count or a misaligned input): padding on every side, including
    runs that would start before the input (the first image's top-left
    corner), strides, vertical dilation, batches, automatic and forced k
    slices, against the oracle element by element."""
    n, h, w, c, k, r, s, stride, pad, dil, x_off = shape
    for split in (-1, 1, 3, 100):
        _check("i16", n, h, w, c, k, r, s, stride, pad, dil, seed=950 + sum(shape[:7]),
               kernel=_kid("i16_small_64x64"), split=split, x_off=x_off)
    _check("i16", n, h, w, c, k, r, s, stride, pad, dil, seed=951 + sum(shape[:7]), x_off=x_off)


def test_small_kernel_gather_preconditions():
    """Output channels not a multiple of 8, misaligned weights, or a filter
    row that is not one input run (horizontal dilation with several columns
    and channels not a multiple of 64): an explicit request for the small
    kernel is refused and Y is left alone."""
    import torch
    ig = _ig()
    for (c, k, x_off, w_off, dw) in ((64, 20, 0, 0, 1), (48, 64, 0, 1, 1), (48, 64, 0, 0, 2)):
        X, W, Y = workloads.random_conv_operands("i16", 1, 6, 6, c, k, 3, 3, 6, 6, 5)
        Xd, Wd = to_device(X, x_off), to_device(W, w_off)
        Yd = torch.from_numpy(Y).cuda()
        d = ig.conv_desc(1, 6, 6, c, k, 3, 3, (1, 1), (1, dw), (1, dw))
        st = ig.igemm_conv2d_ex(2, d, Xd.data_ptr(), Wd.data_ptr(), Yd.data_ptr(),
                                torch.cuda.current_stream().cuda_stream,
                                _kid("i16_small_64x64"), -1)
        torch.cuda.synchronize()
        assert st == ig.IGEMM_EINVAL and np.array_equal(Yd.cpu().numpy(), Y), (c, k, x_off)


@pytest.mark.parametrize("dt", ["i16", "i8"])
@pytest.mark.parametrize("x_off,w_off", [(1, 0), (0, 1), (3, 5)])
def test_misaligned_tensors(dt, x_off, w_off):
    """Bases off 16-byte alignment: element gather for X, element loads of W."""
    for name in CONV_KERNELS[dt]:
        _check(dt, 2, 11, 9, 16, 50, 3, 3, (1, 1), (1, 1), (1, 1), seed=31 + x_off + w_off,
               kernel=_kid(name), x_off=x_off, w_off=w_off)


def test_automatic_plans_on_small_layers():
    """Automatic kernel choice across output sizes (16, 32, 64-row tiles)."""
    for (n, hw, c, k) in ((1, 4, 64, 64), (1, 5, 32, 96), (1, 8, 40, 128), (2, 14, 24, 64),
                          (1, 28, 16, 130)):
        for dt in ("i16", "i8"):
            _check(dt, n, hw, hw, c, k, 3, 3, (1, 1), (1, 1), (1, 1), seed=hw + c)


def test_wraparound_extremes():
    """All-minimum int16 inputs with a deep window: the exact sums exceed
    2^31, so the result checks the modulo-2^32 update."""
    n, h, w, c, k, r, s = 1, 8, 8, 512, 64, 3, 3
    X = np.full((n, h, w, c), -32768, dtype=np.int16)
    W = np.full((r, s, c, k), -32768, dtype=np.int16)
    W[:, :, ::2, ::3] = 32767
    Y = np.full((n, h, w, k), 2 ** 31 - 5, dtype=np.int32)
    for name in CONV_KERNELS["i16"] + ("i16_small_64x64",):
        want = _oracle(X, W, Y, (1, 1), (1, 1), (1, 1))
        got = _gpu(X, W, Y, (1, 1), (1, 1), (1, 1), kernel=_kid(name))
        assert np.array_equal(got, want), _describe(got, want)


def test_zero_channels_and_empty_output_leave_y():
    """k = r*s*c = 0 and a window that never fits are no-ops."""
    import torch
    ig = _ig()
    Y = torch.full((1, 4, 4, 8), 7, dtype=torch.int32, device="cuda")
    d = ig.conv_desc(1, 4, 4, 0, 8, 1, 1)
    assert ig.igemm_conv2d_i16(d, 0, 0, Y.data_ptr()) == 0
    d = ig.conv_desc(1, 2, 2, 4, 8, 3, 3)
    assert ig.igemm_conv2d_i8(d, 0, 0, Y.data_ptr()) == 0
    torch.cuda.synchronize()
    assert bool((Y == 7).all())


def test_tensor_wrapper_matches_oracle():
    """conv2d() on torch tensors, both operand types."""
    import torch
    ig = _ig()
    for dt in ("i16", "i8"):
        X, W, Y = workloads.random_conv_operands(dt, 2, 15, 15, 24, 48, 3, 3, 8, 8, seed=9)
        want = _oracle(X, W, Y, (2, 2), (1, 1), (1, 1))
        Yd = torch.from_numpy(Y).cuda()
        ig.conv2d(torch.from_numpy(X).cuda(), torch.from_numpy(W).cuda(), Yd, stride=(2, 2),
                  pad=(1, 1))
        torch.cuda.synchronize()
        got = Yd.cpu().numpy()
        assert np.array_equal(got, want), _describe(got, want)


def test_graph_replays_match_oracle():
    """A convolution captured in a HIP graph (it uses no workspace and no
    memset): every replay adds conv(X, W) once more, checked after each
    replay, with eager work on the stream between replays."""
    import torch
    ig = _ig()
    X, W, Y = workloads.random_conv_operands("i16", 2, 14, 14, 32, 72, 3, 3, 7, 7, seed=21)
    Xd, Wd, Yd = (torch.from_numpy(a).cuda() for a in (X, W, Y))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ig.conv2d(Xd, Wd, Yd, stride=(2, 2), pad=(1, 1))   # eager call before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    want = _oracle(X, W, Y, (2, 2), (1, 1), (1, 1))
    assert np.array_equal(Yd.cpu().numpy(), want), _describe(Yd.cpu().numpy(), want)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ig.conv2d(Xd, Wd, Yd, stride=(2, 2), pad=(1, 1))
    for rep in range(3):
        g.replay()
        scratch = torch.ones(1 << 16, device="cuda", dtype=torch.int32) * rep  # eager work
        torch.cuda.synchronize()
        want = _oracle(X, W, want, (2, 2), (1, 1), (1, 1))
        got = Yd.cpu().numpy()
        assert np.array_equal(got, want), f"replay {rep}: " + _describe(got, want)
        del scratch


def _fuzz_cases(n_cases=60, seed=4242):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        dt = "i16" if rng.integers(0, 3) else "i8"
        n = int(rng.integers(1, 4))
        r, s = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        st = (int(rng.integers(1, 4)), int(rng.integers(1, 4)))
        dl = (int(rng.integers(1, 4)), int(rng.integers(1, 4)))
        pd = (int(rng.integers(0, 5)), int(rng.integers(0, 5)))
        h = int(rng.integers(1, 24))
        w = int(rng.integers(1, 24))
        c = int(rng.choice([1, 2, 3, 5, 8, 13, 16, 24, 32, 40, 64]))
        k = int(rng.choice([1, 3, 17, 64, 100, 129, 256, 300]))
        kname = str(rng.choice(list(CONV_KERNELS[dt]) + ["auto"]))
        split = int(rng.choice([-1, -1, 1, 2, 3, 7]))
        x_off = int(rng.choice([0, 0, 1, 3]))
        out.append((i, dt, n, h, w, c, k, r, s, st, pd, dl, kname, split, x_off))
    return out


_FUZZ = _fuzz_cases()


@pytest.mark.parametrize("case", _FUZZ, ids=[f"f{c[0]}-{c[1]}-{c[2]}x{c[3]}x{c[4]}x{c[5]}-k{c[6]}"
                                             f"-r{c[7]}s{c[8]}" for c in _FUZZ])
def test_fuzz_conv(case):
    """Seeded random convolutions: batch, extents, channels, filter sizes,
    strides, dilations and padding (windows that do not fit give empty
    outputs), random kernel and k-slice count, misaligned X."""
    i, dt, n, h, w, c, k, r, s, st, pd, dl, kname, split, x_off = case
    ig = _ig()
    oh = ig.igemm_conv2d_out_dim(h, r, st[0], pd[0], dl[0])
    ow = ig.igemm_conv2d_out_dim(w, s, st[1], pd[1], dl[1])
    X, W, Y = workloads.random_conv_operands(dt, n, h, w, c, k, r, s, oh, ow, seed=7000 + i)
    want = _oracle(X, W, Y, st, pd, dl)
    kid = -1 if kname == "auto" else _kid(kname)
    got = _gpu(X, W, Y, st, pd, dl, kernel=kid, split=split, x_off=x_off)
    assert np.array_equal(got, want), _describe(got, want)


def test_window_deeper_than_one_workgroup_range():
    """k = r*s*c = 3*3*4096 = 36864 exceeds the 32768 elements one
    workgroup accumulates, so the lowered GEMM is sliced along k and the
    slices are added atomically; full-range operands make the exact sums
    wrap modulo 2^32. Every conv kernel of both types."""
    for dt in ("i16", "i8"):
        for name in CONV_KERNELS[dt]:
            _check(dt, 1, 3, 4, 4096, 24, 3, 3, (1, 1), (1, 1), (1, 1), seed=88,
                   kernel=_kid(name))
