"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/igemm.h declares, rejects invalid arguments before any HIP
call, and plans launches as documented."""
import ctypes
import os
import re

import pytest

import paper_2302_07594_amd as ig

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "igemm.h")

FAKE_A = 0x10000   # never dereferenced: every call below fails validation or is a no-op
FAKE_B = 0x20000
FAKE_C = 0x30000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(igemm_\w+)\s*\(", text, re.M)))


def test_header_declares_entry_points():
    fns = declared_functions()
    for name in ("igemm_i16", "igemm_i8", "igemm_strerror", "igemm_i16_ex", "igemm_i8_ex",
                 "igemm_query_plan", "igemm_num_kernels", "igemm_kernel_name",
                 "igemm_version", "igemm_i16_ws", "igemm_i8_ws",
                 "igemm_pack_i16", "igemm_pack_i8", "igemm_i16_prepacked",
                 "igemm_i8_prepacked", "igemm_pack_b_i16", "igemm_pack_b_i8",
                 "igemm_i16_packed_b", "igemm_i8_packed_b"):
        assert name in fns


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ig.library_path())
    for name in declared_functions():
        assert hasattr(lib, name), name


def _imported_symbols(path):
    import shutil
    import subprocess
    if shutil.which("nm") is None:
        pytest.skip("nm not available")
    out = subprocess.run(["nm", "-D", "--undefined-only", path], capture_output=True,
                         text=True, check=True).stdout
    return {line.split()[-1].split("@")[0] for line in out.splitlines() if line.strip()}


def test_library_allocates_no_device_memory():
    """The boundary allocates nothing and keeps no pool: the library imports
    no HIP allocation, free, pool, memset or copy routine at all, so no call
    can reach one; its only HIP imports are the launch machinery, the device
    query for the compute-unit count and error reporting."""
    hip = {s for s in _imported_symbols(ig.library_path()) if "hip" in s.lower()}
    forbidden = [s for s in hip if any(w in s for w in
                                       ("Malloc", "Free", "MemPool", "Memset", "Memcpy",
                                        "HostRegister", "StreamCreate", "EventCreate"))]
    assert not forbidden, forbidden
    allowed = {"hipLaunchKernel", "hipGetLastError", "hipGetDevice", "hipDeviceGetAttribute",
               "hipGetSymbolAddress", "__hipPushCallConfiguration",
               "__hipPopCallConfiguration", "__hipRegisterFatBinary", "__hipRegisterFunction",
               "__hipUnregisterFatBinary", "__hipRegisterVar", "__hipRegisterManagedVar"}
    assert hip <= allowed, sorted(hip - allowed)


def test_build_stamp_tracks_sources():
    """The build records the hash of the sources, headers and flags it used;
    the test session's library is current, and any change of flags changes
    the hash."""
    from paper_2302_07594_amd import build as hip_build
    assert hip_build.is_current()
    assert hip_build.source_hash(["-DX"]) != hip_build.source_hash()


def test_source_hash_does_not_depend_on_checkout_location(tmp_path):
    """A copy of the tree elsewhere (the GPU runs work on a copy) hashes the
    same: the stamp and the profile summaries' hashes stay valid there."""
    import shutil
    import subprocess
    import sys
    from paper_2302_07594_amd import build as hip_build
    root = os.path.dirname(os.path.dirname(os.path.abspath(hip_build.__file__)))
    dst = tmp_path / "elsewhere"
    shutil.copytree(os.path.join(root, "paper_2302_07594_amd"), dst / "paper_2302_07594_amd",
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    shutil.copytree(os.path.join(root, "include"), dst / "include")
    code = ("from paper_2302_07594_amd import build as b; "
            "print(b.source_hash(), b.kernel_hash('packed'), b.kernel_hash('direct'))")
    # the copy's package stubs import nothing beyond build.py
    out = subprocess.run([sys.executable, "-c", "import sys; sys.path.insert(0, sys.argv[1]); "
                          + code, str(dst)], capture_output=True, text=True, check=True,
                         cwd=str(tmp_path)).stdout.split()
    assert out == [hip_build.source_hash(), hip_build.kernel_hash("packed"),
                   hip_build.kernel_hash("direct")]


def test_oracle_not_linked_into_library():
    lib = ctypes.CDLL(ig.library_path())
    assert not hasattr(lib, "oracle_igemm_i16")


@pytest.mark.parametrize("fn", [ig.igemm_i16, ig.igemm_i8])
def test_invalid_arguments(fn):
    E = ig.IGEMM_EINVAL
    s = 0
    assert fn(-1, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s) == E
    assert fn(4, -1, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s) == E
    assert fn(4, 4, -1, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s) == E
    assert fn(4, 4, 4, FAKE_A, 3, FAKE_B, 4, FAKE_C, 4, s) == E   # lda < k
    assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 3, FAKE_C, 4, s) == E   # ldb < n
    assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 3, s) == E   # ldc < n
    assert fn(4, 4, 4, 0, 4, FAKE_B, 4, FAKE_C, 4, s) == E        # A NULL
    assert fn(4, 4, 4, FAKE_A, 4, 0, 4, FAKE_C, 4, s) == E        # B NULL
    assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 4, 0, 4, s) == E        # C NULL
    big = 1 << 62
    assert fn(big, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, big, s) == E  # extent overflow


@pytest.mark.parametrize("fn", [ig.igemm_i16, ig.igemm_i8])
def test_noop_calls_return_ok_without_device(fn):
    s = 0
    assert fn(0, 4, 4, 0, 4, 0, 4, 0, 4, s) == ig.IGEMM_OK         # m = 0
    assert fn(4, 0, 4, 0, 4, 0, 4, 0, 4, s) == ig.IGEMM_OK         # n = 0
    assert fn(4, 4, 0, 0, 1, 0, 4, FAKE_C, 4, s) == ig.IGEMM_OK    # k = 0: C unchanged


def test_ex_rejects_mismatched_kernel():
    s = 0
    i8_kernel = ig.kernels_for(1)[0]
    i16_kernel = ig.kernels_for(2)[0]
    assert ig.igemm_i16_ex(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s,
                           i8_kernel, -1) == ig.IGEMM_EINVAL
    assert ig.igemm_i8_ex(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s,
                          i16_kernel, -1) == ig.IGEMM_EINVAL
    assert ig.igemm_i8_ex(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s,
                          ig.igemm_num_kernels(), -1) == ig.IGEMM_EINVAL
    assert ig.igemm_i8_ex(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s, -1, 0) == ig.IGEMM_EINVAL


def test_too_large_is_unsupported():
    s = 0
    n = (1 << 31) + 64
    assert ig.igemm_i8(1, n, 1, FAKE_A, 1, FAKE_B, n, FAKE_C, n, s) == ig.IGEMM_ENOTSUP


def test_strerror_and_names():
    assert ig.igemm_strerror(0) == "success"
    assert "invalid" in ig.igemm_strerror(-1)
    assert ig.igemm_strerror(12345) == "unknown status"
    names = [ig.igemm_kernel_name(i) for i in range(ig.igemm_num_kernels())]
    assert all(names) and len(set(names)) == len(names)
    assert ig.igemm_kernel_name(-1) is None
    assert ig.igemm_version() >= 100


def test_plans_for_workloads():
    import workloads
    for wname in workloads.ORDER:
        for case in workloads.WORKLOADS[wname].cases:
            es = 2 if case.dtype == "i16" else 1
            p = ig.igemm_query_plan(es, case.m, case.n, case.k, FAKE_A, case.k, FAKE_B, case.n,
                                    FAKE_C, case.n)
            assert p["elem_bytes"] == es
            assert p["kernel_name"].startswith("i16" if es == 2 else "i8")
            assert p["split"] >= 1 and p["k_chunk"] % 64 == 0
            assert p["split"] * p["k_chunk"] >= case.k > (p["split"] - 1) * p["k_chunk"]
            assert p["k_chunk"] <= 32768
            if p["packed"] or "direct" in p["kernel_name"]:
                # one launch of `grid` workgroups per k chunk
                assert p["grid"] == p["tiles"]
                assert (p["workspace_bytes"] > 0) == bool(p["packed"])
            else:
                assert p["grid"] == p["tiles"] * p["split"] and p["workspace_bytes"] == 0
            assert p["limb_products"] == (4 if es == 2 else 1)
    big = ig.igemm_query_plan(2, 4096, 4096, 4096, FAKE_A, 4096, FAKE_B, 4096, FAKE_C, 4096)
    assert big["kernel_name"] == "i16_packed_128x128" and big["split"] == 1
    big8 = ig.igemm_query_plan(1, 8192, 8192, 8192, FAKE_A, 8192, FAKE_B, 8192, FAKE_C, 8192)
    assert big8["kernel_name"] == "i8_direct_256x256" and big8["split"] == 1
    assert big8["workspace_bytes"] == 0
    # rows that are not 16-byte multiples, or k not a multiple of 256: packed
    odd8 = ig.igemm_query_plan(1, 8192, 8192, 8200, FAKE_A, 8200, FAKE_B, 8192, FAKE_C, 8192)
    assert odd8["kernel_name"] == "i8_packed_256x256"
    small = ig.igemm_query_plan(2, 256, 256, 256, FAKE_A, 256, FAKE_B, 256, FAKE_C, 256)
    assert not small["packed"] and small["workspace_bytes"] == 0
    # small int16 outputs with aligned rows and whole k-tiles: the small-output
    # kernel, at most four k-tiles per workgroup, slices spread evenly
    for (m, n, k, kt) in ((3136, 64, 576, 3), (3136, 256, 64, 1), (784, 128, 1152, 4),
                          (196, 256, 2304, 4), (49, 512, 4608, 4), (256, 256, 256, 1)):
        p = ig.igemm_query_plan(2, m, n, k, FAKE_A, k, FAKE_B, n, FAKE_C, n)
        assert p["kernel_name"] == "i16_small_64x64", (m, n, k)
        assert p["k_chunk"] == 64 * kt and p["split"] == -(-k // p["k_chunk"])
        assert p["grid"] == p["tiles"] * p["split"] and p["threads"] == 256
    # k not a multiple of 64, or rows not whole 16 bytes: the small kernel's
    # ragged variant (A through registers, vec_a = 0); B's rows must still be
    # whole 16-byte chunks
    for (k, lda) in ((147, 147), (576, 577)):
        p = ig.igemm_query_plan(2, 3136, 64, k, FAKE_A, lda, FAKE_B, 64, FAKE_C, 64)
        assert p["kernel_name"] == "i16_small_64x64" and p["vec_a"] == 0
        assert p["split"] == -(-(-(-k // 64)) // (p["k_chunk"] // 64))
        p = ig.igemm_query_plan(2, 3136, 64, k, FAKE_A, lda, FAKE_B, 65, FAKE_C, 64)
        assert p["kernel_name"] != "i16_small_64x64"


def test_plan_alignment_and_split_rules():
    # odd leading dimension or base -> element path
    p = ig.igemm_query_plan(2, 100, 64, 147, FAKE_A, 147, FAKE_B, 64, FAKE_C, 64)
    assert p["vec_a"] == 0 and p["vec_b"] == 1
    p = ig.igemm_query_plan(1, 100, 64, 128, FAKE_A + 1, 128, FAKE_B, 64, FAKE_C, 64)
    assert p["vec_a"] == 0
    # k beyond the per-workgroup cap forces slices
    p = ig.igemm_query_plan(1, 4096, 4096, 100000, FAKE_A, 100000, FAKE_B, 4096, FAKE_C, 4096)
    assert p["split"] >= 4 and p["k_chunk"] <= 32768
    # explicit split is honoured, clamped to the number of k-tiles
    p = ig.igemm_query_plan(1, 64, 64, 640, FAKE_A, 640, FAKE_B, 64, FAKE_C, 64, split=3)
    assert p["split"] == 3
    p = ig.igemm_query_plan(1, 64, 64, 100, FAKE_A, 100, FAKE_B, 64, FAKE_C, 64, split=50)
    assert p["split"] == 2
    # no-op
    p = ig.igemm_query_plan(1, 64, 64, 0, FAKE_A, 1, FAKE_B, 64, FAKE_C, 64)
    assert p["grid"] == 0 and p["kernel"] == -1


def _kid(name):
    return [i for i in range(ig.igemm_num_kernels()) if ig.igemm_kernel_name(i) == name][0]


def test_packed_workspace_layout():
    """int16: two limb planes of A and of B (rows padded to the tile, k to a
    multiple of 256), row corrections and per-slice column corrections; int8
    skips the copy of an A that is aligned and tile-shaped."""
    p = ig.igemm_query_plan(2, 4096, 4096, 4096, FAKE_A, 4096, FAKE_B, 4096, FAKE_C, 4096)
    planes = 2 * 4096 * 4096
    assert p["workspace_bytes"] >= 2 * planes + 4 * 4096 + 4 * 4096
    assert p["workspace_bytes"] % 256 == 0
    kid = _kid("i8_packed_256x256")
    q = ig.igemm_query_plan(1, 512, 300, 768, FAKE_A, 768, FAKE_B, 300, FAKE_C, 300, kernel=kid)
    assert q["workspace_bytes"] == 512 * 768           # B only: n_pad = 512, k_pad = 768
    q = ig.igemm_query_plan(1, 512, 300, 768, FAKE_A + 1, 768, FAKE_B, 300, FAKE_C, 300,
                            kernel=kid)
    assert q["workspace_bytes"] == 512 * 768 + 512 * 768   # misaligned A is copied too
    q = ig.igemm_query_plan(1, 500, 300, 768, FAKE_A, 768, FAKE_B, 300, FAKE_C, 300, kernel=kid)
    assert q["workspace_bytes"] == 512 * 768 + 512 * 768   # ragged m: A is padded
    # k beyond 32768: one main-kernel launch per 32768-element chunk
    q = ig.igemm_query_plan(2, 300, 200, 70000, FAKE_A, 70000, FAKE_B, 200, FAKE_C, 200,
                            kernel=_kid("i16_packed_128x128"))
    assert q["split"] == 3 and q["k_chunk"] == 32768 and q["packed"] == 1


@pytest.mark.parametrize("es", [2, 1])
def test_packed_workspace_parts(es):
    """The workspace is an A part then a B part; the B part (what pack_b
    fills) depends on n, k and the kernel only, never on m or A."""
    kid = _kid("i16_packed_128x128" if es == 2 else "i8_packed_256x256")
    n, k = 1000, 3000
    bparts = set()
    for m, a in ((1, FAKE_A), (1000, FAKE_A), (4096, FAKE_A + 1), (77, FAKE_A)):
        q = ig.igemm_query_plan(es, m, n, k, a, k, FAKE_B, n, FAKE_C, n, kernel=kid)
        assert q["workspace_bytes"] == q["packed_a_bytes"] + q["packed_b_bytes"]
        assert q["packed_a_bytes"] % 256 == 0 and q["packed_b_bytes"] % 256 == 0
        bparts.add(q["packed_b_bytes"])
    n_pad, k_pad = (1024, 3072) if es == 2 else (1024, 3072)
    corr = 4 * n_pad if es == 2 else 0
    assert bparts == {es * n_pad * k_pad + corr}
    # int8 A that is aligned and tile-shaped needs no A part at all
    if es == 1:
        q = ig.igemm_query_plan(1, 512, n, 3072, FAKE_A, 3072, FAKE_B, n, FAKE_C, n, kernel=kid)
        assert q["packed_a_bytes"] == 0


def test_packed_grid_limits():
    kid = _kid("i16_packed_128x128")
    m = 1 << 25   # more padded rows than one launch can cover with pack_a
    with pytest.raises(ig.IgemmError) as e:
        ig.igemm_query_plan(2, m, 256, 256, FAKE_A, 256, FAKE_B, 256, FAKE_C, 256, kernel=kid)
    assert e.value.status == ig.IGEMM_ENOTSUP


@pytest.mark.parametrize("fn", [ig.igemm_i16_ws, ig.igemm_i8_ws])
def test_ws_rejects_bad_workspace(fn):
    s = 0
    E = ig.IGEMM_EINVAL
    # a misaligned or negative-size workspace is refused before any HIP call
    assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s, -1, -1, 0x40001, 1 << 20) == E
    assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, s, -1, -1, 0x40000, -5) == E
    # argument checks come first, as for the other calls
    assert fn(4, 4, 4, FAKE_A, 3, FAKE_B, 4, FAKE_C, 4, s, -1, -1, 0x40000, 1 << 20) == E
    assert fn(0, 4, 4, 0, 4, 0, 4, 0, 4, s, -1, -1, 0, 0) == ig.IGEMM_OK


def test_strerror_enomem():
    assert "workspace" in ig.igemm_strerror(ig.IGEMM_ENOMEM)


@pytest.mark.parametrize("es", [2, 1])
def test_pack_once_calls_reject_bad_arguments(es):
    """Argument, kernel and workspace checks of the pack-once calls come
    before any HIP call."""
    s = 0
    pk = ig.igemm_pack_i16 if es == 2 else ig.igemm_pack_i8
    mul = ig.igemm_i16_prepacked if es == 2 else ig.igemm_i8_prepacked
    W = 0x40000
    E = ig.IGEMM_EINVAL
    fused = ig.kernels_for(es)[0]
    assert pk(64, 64, 64, FAKE_A, 64, FAKE_B, 64, -1, 0, 1 << 20, s) == E        # no workspace
    assert pk(64, 64, 64, FAKE_A, 64, FAKE_B, 64, -1, W + 16, 1 << 20, s) == E   # misaligned
    assert pk(64, 64, 64, FAKE_A, 64, FAKE_B, 64, fused, W, 1 << 20, s) == E     # fused kernel
    assert pk(64, 64, 64, FAKE_A, 63, FAKE_B, 64, -1, W, 1 << 20, s) == E        # lda < k
    assert pk(64, 64, 64, FAKE_A, 64, FAKE_B, 64, -1, W, 256, s) == ig.IGEMM_ENOMEM
    assert pk(0, 64, 64, FAKE_A, 64, FAKE_B, 64, -1, W, 0, s) == ig.IGEMM_OK      # no-op
    assert mul(64, 64, 64, FAKE_A, 64, FAKE_C, 64, -1, 0, 1 << 20, s) == E
    assert mul(64, 64, 64, FAKE_A, 64, 0, 64, -1, W, 1 << 20, s) == E             # C NULL
    assert mul(64, 64, 64, FAKE_A, 64, FAKE_C, 63, -1, W, 1 << 20, s) == E        # ldc < n
    assert mul(64, 64, 64, FAKE_A, 64, FAKE_C, 64, fused, W, 1 << 20, s) == E
    assert mul(64, 64, 64, FAKE_A, 64, FAKE_C, 64, -1, W, 256, s) == ig.IGEMM_ENOMEM
    assert mul(64, 64, 0, FAKE_A, 1, FAKE_C, 64, -1, W, 0, s) == ig.IGEMM_OK


@pytest.mark.parametrize("es", [2, 1])
def test_packed_b_calls_reject_bad_arguments(es):
    """Argument, kernel and buffer checks of the pack-B-once calls come
    before any HIP call."""
    s = 0
    pk = ig.igemm_pack_b_i16 if es == 2 else ig.igemm_pack_b_i8
    mul = ig.igemm_i16_packed_b if es == 2 else ig.igemm_i8_packed_b
    W, P = 0x40000, 0x80000
    E = ig.IGEMM_EINVAL
    fused = ig.kernels_for(es)[0]
    big = 1 << 24
    assert pk(64, 64, FAKE_B, 64, -1, 0, big, s) == E              # no buffer
    assert pk(64, 64, FAKE_B, 64, -1, P + 64, big, s) == E         # misaligned
    assert pk(64, 64, FAKE_B, 64, fused, P, big, s) == E           # fused kernel
    assert pk(64, 64, FAKE_B, 63, -1, P, big, s) == E              # ldb < n
    assert pk(64, 64, 0, 64, -1, P, big, s) == E                   # B NULL
    assert pk(-1, 64, FAKE_B, 64, -1, P, big, s) == E
    assert pk(64, 64, FAKE_B, 64, -1, P, 256, s) == ig.IGEMM_ENOMEM
    assert pk(0, 64, FAKE_B, 64, -1, P, 0, s) == ig.IGEMM_OK       # no-op
    assert pk(64, 0, 0, 64, -1, P, 0, s) == ig.IGEMM_OK
    assert mul(64, 64, 64, FAKE_A, 64, 0, big, FAKE_C, 64, -1, W, big, s) == E      # no B
    assert mul(64, 64, 64, FAKE_A, 64, P + 16, big, FAKE_C, 64, -1, W, big, s) == E
    assert mul(64, 64, 64, FAKE_A, 64, P, big, FAKE_C, 64, fused, W, big, s) == E
    assert mul(64, 64, 64, FAKE_A, 63, P, big, FAKE_C, 64, -1, W, big, s) == E      # lda < k
    assert mul(64, 64, 64, FAKE_A, 64, P, big, 0, 64, -1, W, big, s) == E           # C NULL
    assert mul(64, 64, 64, FAKE_A, 64, P, big, FAKE_C, 63, -1, W, big, s) == E      # ldc < n
    assert mul(64, 64, 64, FAKE_A, 64, P, big, FAKE_C, 64, -1, W + 8, big, s) == E  # misaligned
    assert mul(64, 64, 64, FAKE_A, 64, P, 256, FAKE_C, 64, -1, W, big, s) == ig.IGEMM_ENOMEM
    assert mul(64, 64, 64, FAKE_A, 64, P, big, FAKE_C, 64, -1, W, 256, s) == ig.IGEMM_ENOMEM
    assert mul(0, 64, 64, FAKE_A, 64, 0, 0, FAKE_C, 64, -1, 0, 0, s) == ig.IGEMM_OK


# ---- convolution entry points -----------------------------------------------

FAKE_X, FAKE_W, FAKE_Y = FAKE_A, FAKE_B, FAKE_C


def _cd(**kw):
    base = dict(n=1, h=8, w=8, c=16, k=32, r=3, s=3, stride=(1, 1), pad=(1, 1), dil=(1, 1))
    base.update(kw)
    return ig.conv_desc(**base)


def test_conv_header_declares_entry_points():
    fns = declared_functions()
    for name in ("igemm_conv2d_i16", "igemm_conv2d_i8", "igemm_conv2d_ex",
                 "igemm_conv2d_query_plan", "igemm_conv2d_out_dim"):
        assert name in fns


def test_conv_out_dim_matches_oracle():
    import oracle
    for size in (0, 1, 2, 5, 7, 56, 224):
        for f in (1, 2, 3, 7):
            for st in (1, 2, 3):
                for pd in (0, 1, 3):
                    for dl in (1, 2):
                        assert ig.igemm_conv2d_out_dim(size, f, st, pd, dl) == \
                            oracle.conv2d_out_dim(size, f, st, pd, dl)
    assert ig.igemm_conv2d_out_dim(224, 7, 2, 3, 1) == 112
    assert ig.igemm_conv2d_out_dim(-1, 3, 1, 0, 1) == -1
    assert ig.igemm_conv2d_out_dim(5, 0, 1, 0, 1) == -1
    assert ig.igemm_conv2d_out_dim(5, 3, 0, 0, 1) == -1
    assert ig.igemm_conv2d_out_dim(5, 3, 1, -1, 1) == -1
    assert ig.igemm_conv2d_out_dim(5, 3, 1, 0, 0) == -1
    big = (1 << 62) + 5
    assert ig.igemm_conv2d_out_dim(8, 3, 1, big, 1) == -1      # 2*pad overflows
    assert ig.igemm_conv2d_out_dim(8, 3, 1, 0, big) == -1      # dil*(r-1) overflows


@pytest.mark.parametrize("es,fn", [(2, ig.igemm_conv2d_i16), (1, ig.igemm_conv2d_i8)])
def test_conv_invalid_arguments(es, fn):
    E = ig.IGEMM_EINVAL
    X, W, Y = FAKE_X, FAKE_W, FAKE_Y
    assert fn(_cd(n=-1), X, W, Y, 0) == E
    assert fn(_cd(h=-1), X, W, Y, 0) == E
    assert fn(_cd(c=-2), X, W, Y, 0) == E
    assert fn(_cd(k=-1), X, W, Y, 0) == E
    assert fn(_cd(r=0), X, W, Y, 0) == E
    assert fn(_cd(s=0), X, W, Y, 0) == E
    assert fn(_cd(stride=(0, 1)), X, W, Y, 0) == E
    assert fn(_cd(stride=(1, 0)), X, W, Y, 0) == E
    assert fn(_cd(pad=(-1, 0)), X, W, Y, 0) == E
    assert fn(_cd(dil=(1, 0)), X, W, Y, 0) == E
    assert fn(_cd(), 0, W, Y, 0) == E
    assert fn(_cd(), X, 0, Y, 0) == E
    assert fn(_cd(), X, W, 0, 0) == E
    assert ig.igemm_conv2d_ex(3, _cd(), X, W, Y, 0) == E              # bad element size
    if es == 2:
        assert fn(_cd(), X + 1, W, Y, 0) == E                        # odd int16 X
    else:
        assert ig.igemm_conv2d_query_plan(1, _cd(), X=X + 1)["vec_a"] == 0
    # kernels the lowering does not use, or of the other operand type (the
    # small-output kernel gathers this 16-channel input as runs)
    for kid in range(ig.igemm_num_kernels()):
        name = ig.igemm_kernel_name(kid)
        conv_ok = name in ("i16_128x128", "i16_64x64", "i16_32x128", "i16_16x128", "i8_32x256",
                           "i8_16x256", "i16_small_64x64")
        ok = conv_ok and name.startswith("i16" if es == 2 else "i8")
        if not ok:
            with pytest.raises(ig.IgemmError):
                ig.igemm_conv2d_query_plan(es, _cd(), kernel=kid)
    with pytest.raises(ig.IgemmError):
        ig.igemm_conv2d_query_plan(es, _cd(), kernel=ig.igemm_num_kernels())
    with pytest.raises(ig.IgemmError):
        ig.igemm_conv2d_query_plan(es, _cd(), split=0)


@pytest.mark.parametrize("fn", [ig.igemm_conv2d_i16, ig.igemm_conv2d_i8])
def test_conv_noop_calls_return_ok_without_device(fn):
    OK = ig.IGEMM_OK
    assert fn(_cd(n=0), 0, 0, 0, 0) == OK
    assert fn(_cd(k=0), 0, 0, 0, 0) == OK
    assert fn(_cd(c=0), 0, 0, FAKE_Y, 0) == OK                  # k = r*s*c = 0: Y unchanged
    assert fn(_cd(h=1, r=3, pad=(0, 0)), 0, 0, 0, 0) == OK      # window never fits: oh = 0
    assert fn(_cd(w=2, s=2, dil=(1, 3), pad=(0, 0)), 0, 0, 0, 0) == OK
    # a huge but empty problem is a no-op, not an overflow
    assert fn(_cd(n=1 << 40, h=1 << 40, w=1 << 40, c=1 << 40, k=0), 0, 0, 0, 0) == OK
    assert ig.igemm_conv2d_query_plan(2, _cd(n=0))["kernel"] == -1


def test_conv_too_large_is_unsupported():
    NS = ig.IGEMM_ENOTSUP
    X, W, Y = FAKE_X, FAKE_W, FAKE_Y
    # input above 2 GiB
    assert ig.igemm_conv2d_i16(_cd(n=1, h=1 << 15, w=1 << 15, c=2, r=1, s=1, pad=(0, 0)),
                               X, W, Y, 0) == NS
    # padded image of 2^30 rows
    assert ig.igemm_conv2d_i8(_cd(h=4, pad=((1 << 29), 1)), X, W, Y, 0) == NS
    # lowered m beyond 2^31
    assert ig.igemm_conv2d_i8(_cd(n=1 << 20, h=64, w=64, c=1, r=1, s=1, pad=(0, 0)),
                              X, W, Y, 0) == NS
    # filter tensor of 2 GiB
    assert ig.igemm_conv2d_i16(_cd(c=1 << 14, k=1 << 14, r=3, s=3), X, W, Y, 0) == NS
    # products beyond int64 are refused, not wrapped
    assert ig.igemm_conv2d_i8(_cd(n=1 << 40, h=1 << 28, w=1 << 28, c=1, r=1, s=1,
                                  pad=(0, 0)), X, W, Y, 0) == NS


def test_conv_plans_match_lowered_gemm():
    """The six layers' plans: the lowered GEMM shapes, no workspace, the
    small-output kernel for every layer (whole 64-channel taps by DMA when the
    channels are a multiple of 64 and the tensors aligned; the 3-channel stem
    as input runs, vec_a = 0), the fused kernels with the 16-byte gather when
    the small kernel does not apply and c * element size is a multiple of 16."""
    import workloads
    for case in workloads.CONV2D_CASES:
        m, n, k = case.gemm_shape()
        d = ig.conv_desc(case.n, case.h, case.w, case.c, case.k, case.r, case.s, case.stride,
                         case.pad, case.dil)
        p = ig.igemm_conv2d_query_plan(2, d)
        assert p["kernel_name"] == "i16_small_64x64", case.name
        assert p["k_chunk"] <= 256
        assert not p["packed"] and p["workspace_bytes"] == 0
        assert p["vec_a"] == (1 if (case.c * 2) % 16 == 0 else 0)
        assert p["split"] * p["k_chunk"] >= k > (p["split"] - 1) * p["k_chunk"]
        bm, bn = (int(x) for x in p["kernel_name"].split("_")[-1].split("x"))
        tiles = -(-m // bm) * -(-n // bn)
        assert p["tiles"] == tiles and p["grid"] == tiles * p["split"]
    d = ig.conv_desc(1, 56, 56, 64, 64, 3, 3, (1, 1), (1, 1), (1, 1))
    assert ig.igemm_conv2d_query_plan(2, d, X=FAKE_X + 2)["vec_a"] == 0   # misaligned X
    assert ig.igemm_conv2d_query_plan(1, d)["kernel_name"] == "i8_32x256"
    d1 = ig.conv_desc(1, 4, 4, 64, 64, 1, 1)
    assert ig.igemm_conv2d_query_plan(1, d1)["kernel_name"] == "i8_16x256"
    assert ig.igemm_conv2d_query_plan(2, d1)["kernel_name"] == "i16_small_64x64"
    assert ig.igemm_conv2d_query_plan(2, d1, X=FAKE_X + 2)["kernel_name"] == "i16_small_64x64"
    # weights whose rows are not whole 16 bytes: the fused kernels
    d2 = ig.conv_desc(1, 4, 4, 64, 60, 1, 1)
    assert ig.igemm_conv2d_query_plan(2, d2, X=FAKE_X + 2)["kernel_name"] == "i16_16x128"


def test_conv_null_descriptor():
    lib = ctypes.CDLL(ig.library_path())
    for name in ("igemm_conv2d_i16", "igemm_conv2d_i8"):
        fn = getattr(lib, name)
        fn.argtypes = [ctypes.c_void_p] * 5
        fn.restype = ctypes.c_int
        assert fn(None, FAKE_X, FAKE_W, FAKE_Y, None) == ig.IGEMM_EINVAL


# ---- int16-output (shift-round-saturate) entry points -------------------------

def test_srs_header_declares_entry_points():
    fns = declared_functions()
    for name in ("igemm_i16_srs", "igemm_i8_srs", "igemm_srs_ex", "igemm_srs_query",
                 "igemm_srs_ws"):
        assert name in fns


def test_srs_query_is_host_only_and_consistent():
    """The workspace query needs no device: the packed path's bytes are the
    packed operands' workspace plus two words per padded row and column and
    block; fused choices need none; invalid arguments raise."""
    P = 1 << 20
    m = n = 4096
    kp = [i for i in ig.kernels_for(2) if ig.igemm_kernel_name(i) == "i16_packed_128x128"][0]
    for k, kc, nblocks in ((290, 0, 1), (290, 290, 1), (4096, 256, 16), (1024, 512, 2)):
        # (the int32 GEMM of k = 1024 takes the direct kernel; the int16-output
        # update still packs)
        plan = ig.igemm_query_plan(2, m, n, k, P, k, P, n, P, n, 256, kernel=kp)
        need = ig.igemm_srs_query(2, m, n, k, P, k, P, n, P, n, kc, 256)
        assert need == plan["workspace_bytes"] + 8 * nblocks * (m + n), (k, kc)
    # fused choices: int8 operands, a small product, blocks of 100, over 64 blocks
    assert ig.igemm_srs_query(1, m, n, 4096, P, 4096, P, n, P, n, 256, 256) == 0
    assert ig.igemm_srs_query(2, 256, 256, 256, P, 256, P, 256, P, 256, 0, 256) == 0
    assert ig.igemm_srs_query(2, m, n, 1000, P, 1000, P, n, P, n, 100, 256) == 0
    assert ig.igemm_srs_query(2, m, n, 20000, P, 20000, P, n, P, n, 256, 256) == 0
    assert ig.igemm_srs_query(2, 0, n, 290, P, 290, P, n, P, n, 0, 256) == 0
    with pytest.raises(ig.IgemmError):
        ig.igemm_srs_query(2, m, n, 290, P, 290, P, n, P, n, -1, 256)
    with pytest.raises(ig.IgemmError):
        ig.igemm_srs_query(3, m, n, 290, P, 290, P, n, P, n, 0, 256)
    kid = [i for i in ig.kernels_for(2) if ig.igemm_kernel_name(i) == "i16_packed_128x128"][0]
    with pytest.raises(ig.IgemmError):   # explicit packed kernel, blocks of 100
        ig.igemm_srs_query(2, m, n, 1000, P, 1000, P, n, P, n, 100, 256, kid)
    assert ig.igemm_srs_query(2, 64, 64, 290, P, 290, P, 64, P, 64, 0, 256, kid) > 0


def test_srs_ws_rejects_bad_workspace_before_any_hip_call():
    E = ig.IGEMM_EINVAL
    a, b, c = FAKE_A, FAKE_B, FAKE_C
    assert ig.igemm_srs_ws(2, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0, -1, 0x1010, 1 << 20) == E
    assert ig.igemm_srs_ws(2, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0, -1, 0x100000, -1) == E
    assert ig.igemm_srs_ws(2, 4, 4, 4, a, 4, b, 4, c, 4, -1, 0, 0, 0, -1, None, 0) == E
    assert ig.igemm_srs_ws(3, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0, -1, None, 0) == E


@pytest.mark.parametrize("fn", [ig.igemm_i16_srs, ig.igemm_i8_srs])
def test_srs_invalid_arguments(fn):
    E = ig.IGEMM_EINVAL
    a, b, c = FAKE_A, FAKE_B, FAKE_C
    assert fn(-1, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0) == E
    assert fn(4, 4, 4, a, 3, b, 4, c, 4, 0, 0, 0, 0) == E          # lda < k
    assert fn(4, 4, 4, a, 4, b, 4, c, 3, 0, 0, 0, 0) == E          # ldc < n
    assert fn(4, 4, 4, 0, 4, b, 4, c, 4, 0, 0, 0, 0) == E          # A NULL
    assert fn(4, 4, 4, a, 4, b, 4, 0, 4, 0, 0, 0, 0) == E          # C NULL
    assert fn(4, 4, 4, a, 4, b, 4, c, 4, -1, 0, 0, 0) == E         # kc < 0
    assert fn(4, 4, 4, a, 4, b, 4, c, 4, 0, -1, 0, 0) == E         # shift < 0
    assert fn(4, 4, 4, a, 4, b, 4, c, 4, 0, 48, 0, 0) == E         # shift > 47
    assert fn(4, 4, 4, a, 4, b, 4, c, 4, 0, 3, 2, 0) == E          # round not 0/1


def test_srs_kernel_choice_is_checked():
    E = ig.IGEMM_EINVAL
    a, b, c = FAKE_A, FAKE_B, FAKE_C
    ok16 = {"i16_128x128", "i16_64x64", "i16_32x128", "i16_16x128",
            "i16_packed_128x128"}  # (the packed kernel needs a device for its workspace)
    ok8 = {"i8_32x256", "i8_16x256"}
    for kid in range(ig.igemm_num_kernels()):
        name = ig.igemm_kernel_name(kid)
        for es, ok in ((2, ok16), (1, ok8)):
            if name not in ok:
                assert ig.igemm_srs_ex(es, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0, kid) == E
    assert ig.igemm_srs_ex(3, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0, -1) == E
    assert ig.igemm_srs_ex(2, 4, 4, 4, a, 4, b, 4, c, 4, 0, 0, 0, 0,
                           ig.igemm_num_kernels()) == E


@pytest.mark.parametrize("fn", [ig.igemm_i16_srs, ig.igemm_i8_srs])
def test_srs_noop_and_unsupported(fn):
    assert fn(0, 4, 4, 0, 4, 0, 4, 0, 4, 0, 0, 0, 0) == ig.IGEMM_OK
    assert fn(4, 0, 4, 0, 4, 0, 4, 0, 4, 0, 0, 0, 0) == ig.IGEMM_OK
    assert fn(4, 4, 0, 0, 1, 0, 4, FAKE_C, 4, 5, 7, 1, 0) == ig.IGEMM_OK   # k = 0: C unchanged
    k = 40000
    # one block beyond 32768 elements: unsupported, nothing enqueued
    assert fn(4, 4, k, FAKE_A, k, FAKE_B, 4, FAKE_C, 4, 0, 0, 0, 0) == ig.IGEMM_ENOTSUP
    assert fn(4, 4, k, FAKE_A, k, FAKE_B, 4, FAKE_C, 4, 32769, 0, 0, 0) == ig.IGEMM_ENOTSUP


def test_planner_rules_for_small_int16_outputs():
    """The measured rules for small int16 products on a 256-unit device:
    aligned operands with whole k-tiles take the small-output kernel, and
    so (its ragged variant) do rows of A that are not whole 16-byte chunks
    and k that ends inside a k-tile, while B's rows are; convolutions whose
    input the small kernel cannot gather follow the fused rules (k slices of
    the 64x64 tiles keep two k-tiles each with the count rounded up)."""
    def plan(m, n, k, lda=None):
        p = ig.igemm_query_plan(2, m, n, k, FAKE_A, lda or k, FAKE_B, n, FAKE_C, n, num_cu=256)
        return ig.igemm_kernel_name(p["kernel"]), p["split"], p["k_chunk"]
    assert plan(3136, 64, 576) == ("i16_small_64x64", 3, 192)
    # rows of A not whole 16 bytes, or k ending inside a k-tile: the ragged
    # variant of the small-output kernel
    assert plan(3136, 64, 576, lda=577) == ("i16_small_64x64", 3, 192)
    assert plan(12544, 64, 147) == ("i16_small_64x64", 1, 192)
    assert plan(3136, 256, 64, lda=65) == ("i16_small_64x64", 1, 64)
    assert plan(100352, 256, 64)[0] == "i16_64x64"      # enough 64x64 tiles to fill the units
    # convolutions: the small-output kernel (whole taps by DMA when the
    # channels are a multiple of 64 and X is 16-byte aligned, else input runs:
    # vec_a = 0), and the fused rules where the weights' rows are not whole
    # 16-byte chunks
    d = ig.conv_desc(1, 56, 56, 64, 256, 1, 1)
    p = ig.igemm_conv2d_query_plan(2, d, num_cu=256)
    assert ig.igemm_kernel_name(p["kernel"]) == "i16_small_64x64" and p["vec_a"] == 1
    p = ig.igemm_conv2d_query_plan(2, d, X=2, num_cu=256)
    assert ig.igemm_kernel_name(p["kernel"]) == "i16_small_64x64" and p["vec_a"] == 0
    p = ig.igemm_conv2d_query_plan(2, d, X=2, W=2, num_cu=256)
    assert ig.igemm_kernel_name(p["kernel"]) == "i16_16x128"
    d = ig.conv_desc(1, 56, 56, 64, 64, 3, 3, pad=(1, 1))
    p = ig.igemm_conv2d_query_plan(2, d, num_cu=256)
    assert (ig.igemm_kernel_name(p["kernel"]), p["split"]) == ("i16_small_64x64", 3)
    p = ig.igemm_conv2d_query_plan(2, d, X=2, num_cu=256)
    assert (ig.igemm_kernel_name(p["kernel"]), p["split"]) == ("i16_small_64x64", 3)
    p = ig.igemm_conv2d_query_plan(2, d, X=2, W=2, num_cu=256)
    assert (ig.igemm_kernel_name(p["kernel"]), p["split"]) == ("i16_64x64", 5)


def test_int16_stream_plan_and_preconditions():
    """The int16 column-per-wave kernel: 64-column blocks, 16- or 32-row
    blocks, slices of 8 (or 4) k-steps; operands that break its
    preconditions are refused when the kernel is asked for."""
    kid = _kid("i16_stream_32x64")
    p = ig.igemm_query_plan(2, 8, 4096, 4096, FAKE_A, 4096, FAKE_B, 4096, FAKE_C, 4096,
                            kernel=kid)
    assert (p["bm"], p["bn"], p["threads"], p["k_chunk"], p["split"]) == (16, 64, 256, 256, 16)
    assert p["tiles"] == 64 and p["grid"] == 1024 and p["workspace_bytes"] == 0
    # the automatic plan takes it for up to 16 rows over wide B when the
    # operands allow it
    auto = ig.igemm_query_plan(2, 8, 4096, 4096, FAKE_A, 4096, FAKE_B, 4096, FAKE_C, 4096)
    assert auto["kernel"] == kid and auto["split"] == 16
    for (m, lda) in ((32, 4096), (8, 4100)):
        auto = ig.igemm_query_plan(2, m, 4096, 4096, FAKE_A, lda, FAKE_B, 4096, FAKE_C, 4096)
        assert auto["kernel"] != kid
    p = ig.igemm_query_plan(2, 33, 1000, 3008, FAKE_A, 3008, FAKE_B, 1000, FAKE_C, 1000,
                            kernel=kid, split=6)
    assert (p["bm"], p["k_chunk"], p["split"], p["tiles"]) == (32, 512, 6, 2 * 16)
    for (m, n, k, a, lda, b, ldb) in ((8, 4096, 4000, FAKE_A, 4000, FAKE_B, 4096),  # k % 64
                                      (8, 4092, 4096, FAKE_A, 4096, FAKE_B, 4092),  # n % 8
                                      (8, 4096, 4096, FAKE_A + 2, 4096, FAKE_B, 4096),
                                      (8, 4096, 4096, FAKE_A, 4100, FAKE_B, 4096),  # lda % 8
                                      (8, 4096, 4096, FAKE_A, 4096, FAKE_B + 8, 4096)):
        with pytest.raises(ig.IgemmError) as e:
            ig.igemm_query_plan(2, m, n, k, a, lda, b, ldb, FAKE_C, n, kernel=kid)
        assert e.value.status == ig.IGEMM_EINVAL
    # an int8 call may not name it
    with pytest.raises(ig.IgemmError):
        ig.igemm_query_plan(1, 8, 4096, 4096, FAKE_A, 4096, FAKE_B, 4096, FAKE_C, 4096,
                            kernel=kid)


def test_int8_stream_ring_plans():
    """17 to 32 int8 rows over 64 to 128 column blocks of B: one k slice per
    compute unit's share (two for 11008 columns), each a long range through
    the ring variant; an explicit split asking for more than 16 k-steps per
    workgroup takes it too."""
    for m in (17, 32):
        p = ig.igemm_query_plan(1, m, 11008, 4096, num_cu=256)
        assert p["kernel_name"] == "i8_stream_32x128"
        assert (p["split"], p["k_chunk"], p["vec_b"], p["grid"]) == (2, 2048, 1, 2 * 86)
    # 8192 columns: four slices of 16 steps (all resident, no ring)
    p = ig.igemm_query_plan(1, 32, 8192, 4096, num_cu=256)
    assert (p["split"], p["k_chunk"], p["vec_b"], p["grid"]) == (4, 1024, 1, 4 * 64)
    for (m, n) in ((8, 11008), (32, 4096), (32, 20000)):
        p = ig.igemm_query_plan(1, m, n, 4096, num_cu=256)
        assert p["k_chunk"] <= 1024, (m, n)
    p = ig.igemm_query_plan(1, 5, 1008, 3000, lda=3008, kernel=_kid("i8_stream_32x128"),
                            split=2)
    assert (p["split"], p["k_chunk"], p["vec_b"]) == (2, 24 * 64, 1)

