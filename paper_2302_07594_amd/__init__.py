"""Python binding for libigemm (integer GEMM C += A.B on MI355X / gfx950).

The functions here marshal arguments into the C ABI of ``include/igemm.h``
with ctypes; every step of the computation runs in the HIP library. PyTorch
is used only to hand over device pointers and the current HIP stream. There
is no CPU fallback: the library is loaded at the first call, and that call
raises ImportError if it is not built (``build`` is importable without it).

Same names as the C ABI:
    igemm_i16(m, n, k, A, lda, B, ldb, C, ldc, stream=None)
    igemm_i8 (m, n, k, A, lda, B, ldb, C, ldc, stream=None)
    igemm_i16_ex / igemm_i8_ex(..., kernel=-1, split=-1)
    igemm_i16_ws / igemm_i8_ws(..., kernel=-1, split=-1, workspace=None,
                               workspace_bytes=0)
    igemm_i16_noalloc(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1,
                      split=-1)
    igemm_pack_i16 / igemm_pack_i8(m, n, k, A, lda, B, ldb, kernel=-1,
                                   workspace, workspace_bytes, stream=None)
    igemm_i16_prepacked / igemm_i8_prepacked(m, n, k, A, lda, C, ldc, kernel=-1,
                                             workspace, workspace_bytes, stream=None)
    igemm_pack_b_i16 / igemm_pack_b_i8(n, k, B, ldb, kernel=-1, packed_b,
                                       packed_b_bytes, stream=None)
    igemm_i16_packed_b / igemm_i8_packed_b(m, n, k, A, lda, packed_b, packed_b_bytes,
                                           C, ldc, kernel=-1, workspace=None,
                                           workspace_bytes=0, stream=None)
    igemm_query_plan(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, num_cu=0,
                     kernel=-1, split=-1) -> dict
    igemm_conv2d_i16 / igemm_conv2d_i8(desc, X, W, Y, stream=None)
    igemm_conv2d_ex(elem_bytes, desc, X, W, Y, stream=None, kernel=-1, split=-1)
    igemm_conv2d_query_plan(elem_bytes, desc, X=None, W=None, Y=None, num_cu=0,
                            kernel=-1, split=-1) -> dict
    igemm_conv2d_out_dim(in, f, stride, pad, dil)
    igemm_i16_srs / igemm_i8_srs(m, n, k, A, lda, B, ldb, C, ldc, kc=0, shift=0,
                                 round_half_up=0, stream=None)
    igemm_srs_ex(elem_bytes, ..., stream=None, kernel=-1)
    igemm_srs_query(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc=0, num_cu=0,
                    kernel=-1) -> workspace bytes
    igemm_srs_ws(elem_bytes, ..., stream=None, kernel=-1, workspace=None,
                 workspace_bytes=0)
    igemm_strerror(status), igemm_kernel_name(i), igemm_num_kernels(),
    igemm_version()
A, B, C may be integer device addresses or torch tensors (their data_ptr()).
Tensor conveniences: gemm_i16(A, B, C) and gemm_i8(A, B, C) take 2-D CUDA
tensors with unit stride along rows and update C in place; gemm_srs(A, B, C,
kc, shift, round_half_up) the same with an int16 C; conv2d(X, W, Y,
stride, pad, dil) takes contiguous NHWC / (r, s, c, k) / NHWC tensors; a workspace the
call needs is taken from torch's caching allocator (so the calls can be
captured into a torch CUDA graph) and recorded on the stream the call runs
on; the library itself allocates nothing.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libigemm.so")

IGEMM_OK = 0
IGEMM_EINVAL = -1
IGEMM_EHIP = -2
IGEMM_ENOTSUP = -3
IGEMM_ENOMEM = -4
IGEMM_ESCRATCH = -5
IGEMM_NOALLOC_SCRATCH_BYTES = 72 << 20


class IgemmError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {igemm_strerror(status)} (status {status})")
        self.status = status


class _Plan(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int), ("elem_bytes", ctypes.c_int),
                ("bm", ctypes.c_int), ("bn", ctypes.c_int), ("bk", ctypes.c_int),
                ("split", ctypes.c_int), ("k_chunk", ctypes.c_int64),
                ("tiles", ctypes.c_int64), ("grid", ctypes.c_int64),
                ("threads", ctypes.c_int), ("vec_a", ctypes.c_int), ("vec_b", ctypes.c_int),
                ("limb_products", ctypes.c_int), ("packed", ctypes.c_int),
                ("workspace_bytes", ctypes.c_int64), ("packed_a_bytes", ctypes.c_int64),
                ("packed_b_bytes", ctypes.c_int64)]


class ConvDesc(ctypes.Structure):
    """igemm_conv2d_desc: input n x h x w x c (NHWC), k output channels,
    r x s filters, strides, zero padding and dilations."""
    _fields_ = [(f, ctypes.c_int64) for f in
                ("n", "h", "w", "c", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
                 "dil_h", "dil_w")]


def conv_desc(n, h, w, c, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1)) -> ConvDesc:
    return ConvDesc(int(n), int(h), int(w), int(c), int(k), int(r), int(s), int(stride[0]),
                    int(stride[1]), int(pad[0]), int(pad[1]), int(dil[0]), int(dil[1]))


def _load():
    # torch ships its own HIP runtime whose DT_NEEDED name differs from the
    # soname this library links against; loading torch first lets the dynamic
    # linker bind both to that one runtime, so torch's streams and allocations
    # are valid handles for this library's launches.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python -m paper_2302_07594_amd.build` (the HIP library has no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    gemm_args = [i64, i64, i64, vp, i64, vp, i64, vp, i64, vp]
    for name in ("igemm_i16", "igemm_i8"):
        getattr(lib, name).argtypes = gemm_args
        getattr(lib, name).restype = ci
        getattr(lib, name + "_ex").argtypes = gemm_args + [ci, ci]
        getattr(lib, name + "_ex").restype = ci
        getattr(lib, name + "_ws").argtypes = gemm_args + [ci, ci, vp, i64]
        getattr(lib, name + "_ws").restype = ci
    lib.igemm_i16_noalloc.argtypes = gemm_args + [ci, ci]
    lib.igemm_i16_noalloc.restype = ci
    for name in ("igemm_pack_i16", "igemm_pack_i8"):
        getattr(lib, name).argtypes = [i64, i64, i64, vp, i64, vp, i64, ci, vp, i64, vp]
        getattr(lib, name).restype = ci
    for name in ("igemm_i16_prepacked", "igemm_i8_prepacked"):
        getattr(lib, name).argtypes = [i64, i64, i64, vp, i64, vp, i64, ci, vp, i64, vp]
        getattr(lib, name).restype = ci
    for name in ("igemm_pack_b_i16", "igemm_pack_b_i8"):
        getattr(lib, name).argtypes = [i64, i64, vp, i64, ci, vp, i64, vp]
        getattr(lib, name).restype = ci
    for name in ("igemm_i16_packed_b", "igemm_i8_packed_b"):
        getattr(lib, name).argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64, ci, vp, i64, vp]
        getattr(lib, name).restype = ci
    cd = ctypes.POINTER(ConvDesc)
    lib.igemm_conv2d_i16.argtypes = [cd, vp, vp, vp, vp]
    lib.igemm_conv2d_i16.restype = ci
    lib.igemm_conv2d_i8.argtypes = [cd, vp, vp, vp, vp]
    lib.igemm_conv2d_i8.restype = ci
    lib.igemm_conv2d_ex.argtypes = [ci, cd, vp, vp, vp, vp, ci, ci]
    lib.igemm_conv2d_ex.restype = ci
    lib.igemm_conv2d_query_plan.argtypes = [ci, cd, vp, vp, vp, ci, ci, ci,
                                            ctypes.POINTER(_Plan)]
    lib.igemm_conv2d_query_plan.restype = ci
    for name in ("igemm_i16_srs", "igemm_i8_srs"):
        getattr(lib, name).argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64, i64, ci, ci, vp]
        getattr(lib, name).restype = ci
    lib.igemm_srs_ex.argtypes = [ci, i64, i64, i64, vp, i64, vp, i64, vp, i64, i64, ci, ci, vp,
                                 ci]
    lib.igemm_srs_ex.restype = ci
    lib.igemm_srs_query.argtypes = [ci, i64, i64, i64, vp, i64, vp, i64, vp, i64, i64, ci, ci,
                                    ctypes.POINTER(i64)]
    lib.igemm_srs_query.restype = ci
    lib.igemm_srs_ws.argtypes = [ci, i64, i64, i64, vp, i64, vp, i64, vp, i64, i64, ci, ci, vp,
                                 ci, vp, i64]
    lib.igemm_srs_ws.restype = ci
    lib.igemm_conv2d_out_dim.argtypes = [i64] * 5
    lib.igemm_conv2d_out_dim.restype = i64
    lib.igemm_query_plan.argtypes = [ci, i64, i64, i64, vp, i64, vp, i64, vp, i64, ci, ci, ci,
                                     ctypes.POINTER(_Plan)]
    lib.igemm_query_plan.restype = ci
    lib.igemm_strerror.argtypes = [ci]
    lib.igemm_strerror.restype = ctypes.c_char_p
    lib.igemm_kernel_name.argtypes = [ci]
    lib.igemm_kernel_name.restype = ctypes.c_char_p
    lib.igemm_num_kernels.argtypes = []
    lib.igemm_num_kernels.restype = ci
    lib.igemm_version.argtypes = []
    lib.igemm_version.restype = ci
    return lib


class _Lazy:
    """Loads libigemm.so on first attribute access."""
    _handle = None

    def __getattr__(self, name):
        if _Lazy._handle is None:
            _Lazy._handle = _load()
        return getattr(_Lazy._handle, name)


_lib = _Lazy()


def load() -> None:
    """Load the HIP library now (raises ImportError if it is not built)."""
    if _Lazy._handle is None:
        _Lazy._handle = _load()


def library_path() -> str:
    return LIB_PATH


def _addr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return int(x.data_ptr())
    raise TypeError(f"expected a device address or a tensor, got {type(x).__name__}")


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    if hasattr(stream, "cuda_stream"):
        return int(stream.cuda_stream)
    raise TypeError("stream must be None, an int handle or a torch stream")


def _call(name, m, n, k, A, lda, B, ldb, C, ldc, stream, *extra) -> int:
    fn = getattr(_lib, name)
    st = fn(int(m), int(n), int(k), _addr(A), int(lda), _addr(B), int(ldb), _addr(C), int(ldc),
            _stream(stream), *extra)
    return int(st)


def igemm_i16(m, n, k, A, lda, B, ldb, C, ldc, stream=None) -> int:
    """C += A.B, int16 operands, int32 wraparound C. Returns the status."""
    return _call("igemm_i16", m, n, k, A, lda, B, ldb, C, ldc, stream)


def igemm_i8(m, n, k, A, lda, B, ldb, C, ldc, stream=None) -> int:
    """C += A.B, int8 operands, int32 wraparound C. Returns the status."""
    return _call("igemm_i8", m, n, k, A, lda, B, ldb, C, ldc, stream)


def igemm_i16_ex(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1, split=-1) -> int:
    return _call("igemm_i16_ex", m, n, k, A, lda, B, ldb, C, ldc, stream, int(kernel), int(split))


def igemm_i8_ex(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1, split=-1) -> int:
    return _call("igemm_i8_ex", m, n, k, A, lda, B, ldb, C, ldc, stream, int(kernel), int(split))


def igemm_i16_ws(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1, split=-1,
                 workspace=None, workspace_bytes=0) -> int:
    return _call("igemm_i16_ws", m, n, k, A, lda, B, ldb, C, ldc, stream, int(kernel),
                 int(split), _addr(workspace), int(workspace_bytes))


def igemm_i8_ws(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1, split=-1,
                workspace=None, workspace_bytes=0) -> int:
    return _call("igemm_i8_ws", m, n, k, A, lda, B, ldb, C, ldc, stream, int(kernel),
                 int(split), _addr(workspace), int(workspace_bytes))


def igemm_i16_noalloc(m, n, k, A, lda, B, ldb, C, ldc, stream=None, kernel=-1,
                      split=-1) -> int:
    """igemm_i16_ws with the library's static scratch array as the workspace
    (no allocation; calls that overlap on one GPU race). Returns the status."""
    return _call("igemm_i16_noalloc", m, n, k, A, lda, B, ldb, C, ldc, stream, int(kernel),
                 int(split))


def igemm_pack_i16(m, n, k, A, lda, B, ldb, kernel=-1, workspace=None, workspace_bytes=0,
                   stream=None) -> int:
    return int(_lib.igemm_pack_i16(int(m), int(n), int(k), _addr(A), int(lda), _addr(B),
                                   int(ldb), int(kernel), _addr(workspace), int(workspace_bytes),
                                   _stream(stream)))


def igemm_pack_i8(m, n, k, A, lda, B, ldb, kernel=-1, workspace=None, workspace_bytes=0,
                  stream=None) -> int:
    return int(_lib.igemm_pack_i8(int(m), int(n), int(k), _addr(A), int(lda), _addr(B),
                                  int(ldb), int(kernel), _addr(workspace), int(workspace_bytes),
                                  _stream(stream)))


def igemm_i16_prepacked(m, n, k, A, lda, C, ldc, kernel=-1, workspace=None, workspace_bytes=0,
                        stream=None) -> int:
    return int(_lib.igemm_i16_prepacked(int(m), int(n), int(k), _addr(A), int(lda), _addr(C),
                                        int(ldc), int(kernel), _addr(workspace),
                                        int(workspace_bytes), _stream(stream)))


def igemm_i8_prepacked(m, n, k, A, lda, C, ldc, kernel=-1, workspace=None, workspace_bytes=0,
                       stream=None) -> int:
    return int(_lib.igemm_i8_prepacked(int(m), int(n), int(k), _addr(A), int(lda), _addr(C),
                                       int(ldc), int(kernel), _addr(workspace),
                                       int(workspace_bytes), _stream(stream)))


def igemm_pack_b_i16(n, k, B, ldb, kernel=-1, packed_b=None, packed_b_bytes=0,
                     stream=None) -> int:
    return int(_lib.igemm_pack_b_i16(int(n), int(k), _addr(B), int(ldb), int(kernel),
                                     _addr(packed_b), int(packed_b_bytes), _stream(stream)))


def igemm_pack_b_i8(n, k, B, ldb, kernel=-1, packed_b=None, packed_b_bytes=0,
                    stream=None) -> int:
    return int(_lib.igemm_pack_b_i8(int(n), int(k), _addr(B), int(ldb), int(kernel),
                                    _addr(packed_b), int(packed_b_bytes), _stream(stream)))


def igemm_i16_packed_b(m, n, k, A, lda, packed_b, packed_b_bytes, C, ldc, kernel=-1,
                       workspace=None, workspace_bytes=0, stream=None) -> int:
    return int(_lib.igemm_i16_packed_b(int(m), int(n), int(k), _addr(A), int(lda),
                                       _addr(packed_b), int(packed_b_bytes), _addr(C), int(ldc),
                                       int(kernel), _addr(workspace), int(workspace_bytes),
                                       _stream(stream)))


def igemm_i8_packed_b(m, n, k, A, lda, packed_b, packed_b_bytes, C, ldc, kernel=-1,
                      workspace=None, workspace_bytes=0, stream=None) -> int:
    return int(_lib.igemm_i8_packed_b(int(m), int(n), int(k), _addr(A), int(lda),
                                      _addr(packed_b), int(packed_b_bytes), _addr(C), int(ldc),
                                      int(kernel), _addr(workspace), int(workspace_bytes),
                                      _stream(stream)))


_PLACEHOLDER = 1 << 12  # aligned, non-NULL; the planner never dereferences it


def igemm_query_plan(elem_bytes, m, n, k, A=None, lda=None, B=None, ldb=None, C=None,
                     ldc=None, num_cu=0, kernel=-1, split=-1):
    """The launch the library would make (host-only). Returns a dict, or
    raises IgemmError for invalid arguments. Omitted pointers stand for
    16-byte aligned buffers."""
    A = _PLACEHOLDER if A is None else A
    B = _PLACEHOLDER if B is None else B
    C = _PLACEHOLDER if C is None else C
    lda = k if lda is None else lda
    ldb = n if ldb is None else ldb
    ldc = n if ldc is None else ldc
    p = _Plan()
    st = _lib.igemm_query_plan(int(elem_bytes), int(m), int(n), int(k), _addr(A), int(lda),
                               _addr(B), int(ldb), _addr(C), int(ldc), int(num_cu), int(kernel),
                               int(split), ctypes.byref(p))
    if st != IGEMM_OK:
        raise IgemmError(st, "igemm_query_plan")
    d = {f: getattr(p, f) for f, _ in _Plan._fields_}
    d["kernel_name"] = igemm_kernel_name(p.kernel) if p.kernel >= 0 else None
    return d


def igemm_strerror(status: int) -> str:
    return _lib.igemm_strerror(int(status)).decode()


def igemm_kernel_name(kernel: int):
    r = _lib.igemm_kernel_name(int(kernel))
    return r.decode() if r is not None else None


def igemm_num_kernels() -> int:
    return int(_lib.igemm_num_kernels())


def igemm_version() -> int:
    return int(_lib.igemm_version())


def kernels_for(elem_bytes: int):
    """Indices of the kernels that take operands of ``elem_bytes`` bytes."""
    out = []
    for i in range(igemm_num_kernels()):
        nm = igemm_kernel_name(i)
        if (elem_bytes == 2) == nm.startswith("i16"):
            out.append(i)
    return out


def _check_tensors(A, B, C, torch_dtype, name):
    import torch
    if A.dtype != torch_dtype or B.dtype != torch_dtype:
        raise TypeError(f"{name}: A and B must be {torch_dtype}")
    if C.dtype != torch.int32:
        raise TypeError(f"{name}: C must be torch.int32")
    if A.dim() != 2 or B.dim() != 2 or C.dim() != 2:
        raise ValueError(f"{name}: A, B and C must be 2-D")
    m, k = A.shape
    k2, n = B.shape
    if k2 != k or tuple(C.shape) != (m, n):
        raise ValueError(f"{name}: shapes {tuple(A.shape)} x {tuple(B.shape)} -> {tuple(C.shape)}")
    for t, nm in ((A, "A"), (B, "B"), (C, "C")):
        if not t.is_cuda:
            raise ValueError(f"{name}: {nm} must be a CUDA (HIP) tensor")
        if t.shape[1] > 1 and t.stride(1) != 1:
            raise ValueError(f"{name}: {nm} must have unit stride along rows")

    def ld(t):
        return t.stride(0) if t.shape[0] > 1 else max(t.shape[1], 1)
    return m, n, k, ld(A), ld(B), ld(C)


_num_cu_cache = {}


def _num_cu(device) -> int:
    import torch
    idx = device.index if device.index is not None else torch.cuda.current_device()
    if idx not in _num_cu_cache:
        _num_cu_cache[idx] = torch.cuda.get_device_properties(idx).multi_processor_count
    return _num_cu_cache[idx]


def _aligned_workspace(nbytes, device, stream=None):
    """A uint8 device tensor of nbytes from torch's caching allocator,
    256-byte aligned. It is allocated on torch's current stream and recorded
    on `stream` when the call runs elsewhere (a torch stream, or a raw HIP
    stream handle, wrapped as an external stream), so that the allocator does
    not hand its memory to other work before the call's kernels are done."""
    import torch
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    if stream is not None:
        if isinstance(stream, int):
            if stream != int(torch.cuda.current_stream(device).cuda_stream):
                ws.record_stream(torch.cuda.ExternalStream(stream, device=device))
        elif hasattr(stream, "cuda_stream"):
            ws.record_stream(stream)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + nbytes]


def _gemm(es, A, B, C, stream, kernel, split, workspace, name):
    import torch
    m, n, k, lda, ldb, ldc = _check_tensors(A, B, C, torch.int16 if es == 2 else torch.int8, name)
    fn = igemm_i16_ws if es == 2 else igemm_i8_ws
    ws, ws_bytes = None, 0
    if workspace is None or workspace == "torch":
        if m and n and k:
            plan = igemm_query_plan(es, m, n, k, A, lda, B, ldb, C, ldc, _num_cu(C.device),
                                    kernel, split)
            if plan["workspace_bytes"] > 0:
                ws_bytes = plan["workspace_bytes"]
                ws = _aligned_workspace(ws_bytes, C.device, stream)
    elif workspace == "none":
        pass
    elif hasattr(workspace, "data_ptr"):
        ws, ws_bytes = workspace, workspace.numel() * workspace.element_size()
    else:
        raise ValueError(f"{name}: workspace must be None, 'torch', 'none' or a tensor")
    st = fn(m, n, k, A, lda, B, ldb, C, ldc, stream, kernel, split, ws, ws_bytes)
    if st != IGEMM_OK:
        raise IgemmError(st, name)
    return C


class Packed:
    """Packed operands of C += A.B (pack once, multiply many times).

    Holds the device workspace written by igemm_pack_*, the shape and the A
    it was packed with (int8 plans may read A in place)."""

    def __init__(self, es, m, n, k, A, lda, kernel, workspace, nbytes):
        self.es, self.m, self.n, self.k = es, m, n, k
        self.A, self.lda, self.kernel = A, lda, kernel
        self.workspace, self.nbytes = workspace, nbytes


def _packed_kernel(es):
    want = "i16_packed_128x128" if es == 2 else "i8_packed_256x256"
    return [i for i in range(igemm_num_kernels()) if igemm_kernel_name(i) == want][0]


def pack(A, B, stream=None):
    """Pack the operands of C += A.B (2-D torch.int16 or torch.int8 CUDA
    tensors, unit stride along rows). Returns a Packed object for
    gemm_prepacked; A must stay alive and unchanged while it is used."""
    import torch
    if A.dtype not in (torch.int16, torch.int8) or B.dtype != A.dtype:
        raise TypeError("pack: A and B must both be torch.int16 or both torch.int8")
    es = 2 if A.dtype == torch.int16 else 1
    if A.dim() != 2 or B.dim() != 2 or A.shape[1] != B.shape[0]:
        raise ValueError(f"pack: shapes {tuple(A.shape)} x {tuple(B.shape)}")
    for t, nm in ((A, "A"), (B, "B")):
        if not t.is_cuda:
            raise ValueError(f"pack: {nm} must be a CUDA (HIP) tensor")
        if t.shape[1] > 1 and t.stride(1) != 1:
            raise ValueError(f"pack: {nm} must have unit stride along rows")
    m, k = A.shape
    n = B.shape[1]
    lda = A.stride(0) if m > 1 else max(k, 1)
    ldb = B.stride(0) if k > 1 else max(n, 1)
    kid = _packed_kernel(es)
    nbytes = 0
    if m and n and k:
        plan = igemm_query_plan(es, m, n, k, A, lda, B, ldb, None, n, _num_cu(A.device), kid)
        nbytes = plan["workspace_bytes"]
    ws = _aligned_workspace(max(nbytes, 1), A.device, stream)
    fn = igemm_pack_i16 if es == 2 else igemm_pack_i8
    st = fn(m, n, k, A, lda, B, ldb, kid, ws, nbytes, stream)
    if st != IGEMM_OK:
        raise IgemmError(st, "pack")
    return Packed(es, m, n, k, A, lda, kid, ws, nbytes)


def gemm_prepacked(P, C, stream=None):
    """C += A.B from operands packed by pack(); C is a torch.int32 CUDA
    tensor of shape (m, n) with unit stride along rows. Returns C."""
    import torch
    if C.dtype != torch.int32 or C.dim() != 2 or tuple(C.shape) != (P.m, P.n) or not C.is_cuda:
        raise ValueError("gemm_prepacked: C must be an int32 CUDA tensor of shape (m, n)")
    if C.shape[1] > 1 and C.stride(1) != 1:
        raise ValueError("gemm_prepacked: C must have unit stride along rows")
    ldc = C.stride(0) if C.shape[0] > 1 else max(C.shape[1], 1)
    fn = igemm_i16_prepacked if P.es == 2 else igemm_i8_prepacked
    st = fn(P.m, P.n, P.k, P.A, P.lda, C, ldc, P.kernel, P.workspace, P.nbytes, stream)
    if st != IGEMM_OK:
        raise IgemmError(st, "gemm_prepacked")
    return C


class PackedB:
    """The fixed operand B of C += A.B in packed form (pack once, multiply
    with any A of k columns). Holds the device buffer igemm_pack_b_* wrote."""

    def __init__(self, es, n, k, kernel, buf, nbytes):
        self.es, self.n, self.k, self.kernel = es, n, k, kernel
        self.buf, self.nbytes = buf, nbytes


def pack_b(B, stream=None):
    """Pack a 2-D torch.int16 or torch.int8 CUDA tensor B (k x n, unit stride
    along rows) for gemm_packed_b. Returns a PackedB."""
    import torch
    if B.dtype not in (torch.int16, torch.int8) or B.dim() != 2 or not B.is_cuda:
        raise TypeError("pack_b: B must be a 2-D torch.int16 or torch.int8 CUDA tensor")
    if B.shape[1] > 1 and B.stride(1) != 1:
        raise ValueError("pack_b: B must have unit stride along rows")
    es = 2 if B.dtype == torch.int16 else 1
    k, n = B.shape
    ldb = B.stride(0) if k > 1 else max(n, 1)
    kid = _packed_kernel(es)
    nbytes = 0
    if n and k:
        nbytes = igemm_query_plan(es, 1, n, k, None, k, B, ldb, None, n, _num_cu(B.device),
                                  kid)["packed_b_bytes"]
    buf = _aligned_workspace(max(nbytes, 1), B.device, stream)
    fn = igemm_pack_b_i16 if es == 2 else igemm_pack_b_i8
    st = fn(n, k, B, ldb, kid, buf, nbytes, stream)
    if st != IGEMM_OK:
        raise IgemmError(st, "pack_b")
    return PackedB(es, n, k, kid, buf, nbytes)


def gemm_packed_b(A, PB, C, stream=None):
    """C += A.B with B packed by pack_b: A is an m x k CUDA tensor of B's
    type, C an m x n torch.int32 CUDA tensor (unit stride along rows).
    A's packed copy takes memory from torch's caching allocator. Returns C."""
    import torch
    want = torch.int16 if PB.es == 2 else torch.int8
    if A.dtype != want or A.dim() != 2 or A.shape[1] != PB.k or not A.is_cuda:
        raise ValueError(f"gemm_packed_b: A must be a {want} CUDA tensor with {PB.k} columns")
    m = A.shape[0]
    if C.dtype != torch.int32 or C.dim() != 2 or tuple(C.shape) != (m, PB.n) or not C.is_cuda:
        raise ValueError("gemm_packed_b: C must be an int32 CUDA tensor of shape (m, n)")
    for t, nm in ((A, "A"), (C, "C")):
        if t.shape[1] > 1 and t.stride(1) != 1:
            raise ValueError(f"gemm_packed_b: {nm} must have unit stride along rows")
    lda = A.stride(0) if m > 1 else max(PB.k, 1)
    ldc = C.stride(0) if m > 1 else max(PB.n, 1)
    ws, ws_bytes = None, 0
    if m and PB.n and PB.k:
        ws_bytes = igemm_query_plan(PB.es, m, PB.n, PB.k, A, lda, None, PB.n, C, ldc,
                                    _num_cu(C.device), PB.kernel)["packed_a_bytes"]
        if ws_bytes > 0:
            ws = _aligned_workspace(ws_bytes, C.device, stream)
    fn = igemm_i16_packed_b if PB.es == 2 else igemm_i8_packed_b
    st = fn(m, PB.n, PB.k, A, lda, PB.buf, PB.nbytes, C, ldc, PB.kernel, ws, ws_bytes, stream)
    if st != IGEMM_OK:
        raise IgemmError(st, "gemm_packed_b")
    return C


def gemm_i16(A, B, C, stream=None, kernel=-1, split=-1, workspace=None):
    """C += A.B for 2-D torch.int16 CUDA tensors A (m x k), B (k x n) and a
    torch.int32 C (m x n). Returns C. Raises IgemmError on a bad status.
    workspace: None / "torch" (a workspace from torch's allocator when the
    plan packs the operands), "none" (no workspace: the in-place kernels
    only) or a uint8 CUDA tensor (256-byte aligned) to use as is."""
    return _gemm(2, A, B, C, stream, kernel, split, workspace, "gemm_i16")


def gemm_i8(A, B, C, stream=None, kernel=-1, split=-1, workspace=None):
    """C += A.B for 2-D torch.int8 CUDA tensors; see gemm_i16."""
    return _gemm(1, A, B, C, stream, kernel, split, workspace, "gemm_i8")


# ---- int16-output update (shift-round-saturate per k block) -----------------

def igemm_i16_srs(m, n, k, A, lda, B, ldb, C, ldc, kc=0, shift=0, round_half_up=0,
                  stream=None) -> int:
    """int16 C += srs(A B) per k block (see include/igemm.h). Returns the status."""
    return int(_lib.igemm_i16_srs(m, n, k, _addr(A), lda, _addr(B), ldb, _addr(C), ldc, kc,
                                  int(shift), int(round_half_up), _stream(stream)))


def igemm_i8_srs(m, n, k, A, lda, B, ldb, C, ldc, kc=0, shift=0, round_half_up=0,
                 stream=None) -> int:
    return int(_lib.igemm_i8_srs(m, n, k, _addr(A), lda, _addr(B), ldb, _addr(C), ldc, kc,
                                 int(shift), int(round_half_up), _stream(stream)))


def igemm_srs_ex(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc=0, shift=0, round_half_up=0,
                 stream=None, kernel=-1) -> int:
    return int(_lib.igemm_srs_ex(int(elem_bytes), m, n, k, _addr(A), lda, _addr(B), ldb,
                                 _addr(C), ldc, kc, int(shift), int(round_half_up),
                                 _stream(stream), int(kernel)))


def igemm_srs_query(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc=0, num_cu=0,
                    kernel=-1) -> int:
    """Workspace bytes igemm_srs_ws needs for these arguments (0: fused
    path). Host only. Raises IgemmError for invalid arguments."""
    out = ctypes.c_int64(0)
    st = int(_lib.igemm_srs_query(int(elem_bytes), m, n, k, _addr(A), lda, _addr(B), ldb,
                                  _addr(C), ldc, kc, int(num_cu), int(kernel), ctypes.byref(out)))
    if st != IGEMM_OK:
        raise IgemmError(st, "igemm_srs_query")
    return int(out.value)


def igemm_srs_ws(elem_bytes, m, n, k, A, lda, B, ldb, C, ldc, kc=0, shift=0, round_half_up=0,
                 stream=None, kernel=-1, workspace=None, workspace_bytes=0) -> int:
    return int(_lib.igemm_srs_ws(int(elem_bytes), m, n, k, _addr(A), lda, _addr(B), ldb,
                                 _addr(C), ldc, kc, int(shift), int(round_half_up),
                                 _stream(stream), int(kernel),
                                 _addr(workspace) if workspace is not None else None,
                                 int(workspace_bytes)))


def gemm_srs(A, B, C, kc=0, shift=0, round_half_up=False, stream=None, kernel=-1,
             workspace=None):
    """int16 C += srs(A B) for 2-D CUDA tensors: A (m x k) and B (k x n) both
    torch.int16 or both torch.int8, C (m x n) torch.int16, rows with unit
    stride. Per block of kc k indices (0: all of k) the exact product is
    shifted right by `shift` (floor, or round-half-up), saturated to int16
    and added to C modulo 2^16. `workspace` as for gemm_i16: None or 'torch'
    (a workspace from torch's allocator when the packed path is taken, so the
    call may be captured into a graph), 'none' (fused kernels only) or a
    uint8 tensor. Returns C."""
    import torch
    if A.dtype not in (torch.int16, torch.int8) or B.dtype != A.dtype:
        raise TypeError("gemm_srs: A and B must both be torch.int16 or both torch.int8")
    if C.dtype != torch.int16:
        raise TypeError("gemm_srs: C must be torch.int16")
    # the shared checks expect an int32 C: check a stand-in of C's shape
    stand_in = torch.empty_strided(C.shape, C.stride(), dtype=torch.int32, device=C.device)
    m, n, k, lda, ldb, ldc = _check_tensors(A, B, stand_in, A.dtype, "gemm_srs")
    es = 2 if A.dtype == torch.int16 else 1
    ws, ws_bytes = None, 0
    if workspace is None or workspace == "torch":
        if m and n and k:
            ws_bytes = igemm_srs_query(es, m, n, k, A, lda, B, ldb, C, ldc, kc,
                                       _num_cu(C.device), kernel)
            if ws_bytes > 0:
                ws = _aligned_workspace(ws_bytes, C.device, stream)
    elif workspace == "none":
        pass
    elif hasattr(workspace, "data_ptr"):
        ws, ws_bytes = workspace, workspace.numel() * workspace.element_size()
    else:
        raise ValueError("gemm_srs: workspace must be None, 'torch', 'none' or a tensor")
    st = igemm_srs_ws(es, m, n, k, A, lda, B, ldb, C, ldc, kc, shift,
                      1 if round_half_up else 0, stream, kernel, ws, ws_bytes)
    if st != IGEMM_OK:
        raise IgemmError(st, "gemm_srs")
    return C


# ---- convolution through its IM2ROW lowering --------------------------------

def igemm_conv2d_out_dim(size, f, stride=1, pad=0, dil=1) -> int:
    return int(_lib.igemm_conv2d_out_dim(int(size), int(f), int(stride), int(pad), int(dil)))


def igemm_conv2d_i16(desc, X, W, Y, stream=None) -> int:
    """Y += conv(X, W), int16 operands (see include/igemm.h). Returns the status."""
    return int(_lib.igemm_conv2d_i16(ctypes.byref(desc), _addr(X), _addr(W), _addr(Y),
                                     _stream(stream)))


def igemm_conv2d_i8(desc, X, W, Y, stream=None) -> int:
    return int(_lib.igemm_conv2d_i8(ctypes.byref(desc), _addr(X), _addr(W), _addr(Y),
                                    _stream(stream)))


def igemm_conv2d_ex(elem_bytes, desc, X, W, Y, stream=None, kernel=-1, split=-1) -> int:
    return int(_lib.igemm_conv2d_ex(int(elem_bytes), ctypes.byref(desc), _addr(X), _addr(W),
                                    _addr(Y), _stream(stream), int(kernel), int(split)))


def igemm_conv2d_query_plan(elem_bytes, desc, X=None, W=None, Y=None, num_cu=0, kernel=-1,
                            split=-1) -> dict:
    """Plan of the lowered GEMM (host-only); omitted pointers stand for
    16-byte aligned buffers."""
    p = _Plan()
    st = _lib.igemm_conv2d_query_plan(
        int(elem_bytes), ctypes.byref(desc), _addr(_PLACEHOLDER if X is None else X),
        _addr(_PLACEHOLDER if W is None else W), _addr(_PLACEHOLDER if Y is None else Y),
        int(num_cu), int(kernel), int(split), ctypes.byref(p))
    if st != IGEMM_OK:
        raise IgemmError(st, "igemm_conv2d_query_plan")
    d = {f: getattr(p, f) for f, _ in _Plan._fields_}
    d["kernel_name"] = igemm_kernel_name(p.kernel) if p.kernel >= 0 else None
    return d


def conv2d(X, W, Y, stride=(1, 1), pad=(0, 0), dil=(1, 1), stream=None, kernel=-1, split=-1):
    """Y += conv(X, W) on contiguous CUDA tensors: X n x h x w x c and W
    r x s x c x k (both torch.int16 or both torch.int8), Y n x oh x ow x k
    torch.int32. Returns Y; raises IgemmError on a bad status."""
    import torch
    if X.dtype not in (torch.int16, torch.int8) or W.dtype != X.dtype:
        raise TypeError("conv2d: X and W must both be torch.int16 or both torch.int8")
    if Y.dtype != torch.int32:
        raise TypeError("conv2d: Y must be torch.int32")
    for t, nm in ((X, "X"), (W, "W"), (Y, "Y")):
        if t.dim() != 4 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError(f"conv2d: {nm} must be a contiguous 4-D CUDA tensor")
    n, h, w, c = X.shape
    r, s, c2, k = W.shape
    oh = igemm_conv2d_out_dim(h, r, stride[0], pad[0], dil[0])
    ow = igemm_conv2d_out_dim(w, s, stride[1], pad[1], dil[1])
    if c2 != c or tuple(Y.shape) != (n, oh, ow, k):
        raise ValueError(f"conv2d: X {tuple(X.shape)}, W {tuple(W.shape)} need Y "
                         f"{(n, oh, ow, k)}, got {tuple(Y.shape)}")
    d = conv_desc(n, h, w, c, k, r, s, stride, pad, dil)
    st = igemm_conv2d_ex(2 if X.dtype == torch.int16 else 1, d, X, W, Y, stream, kernel, split)
    if st != IGEMM_OK:
        raise IgemmError(st, "conv2d")
    return Y
