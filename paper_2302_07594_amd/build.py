"""Build the HIP library ``libigemm.so`` for gfx950, in-tree.

``python -m paper_2302_07594_amd.build`` (or ``build()``) compiles
``csrc/*.hip`` and ``csrc/*.cpp`` with hipcc into
``paper_2302_07594_amd/libigemm.so``. The library exports the C ABI declared
in ``include/igemm.h``.

Next to the library, ``libigemm.so.sha256`` records the SHA-256 of every
source, header and compiler flag the library was built from
(``source_hash()``); ``is_current()`` compares it with the tree, so that
tests can rebuild a library that is out of date instead of running it.
"""
from __future__ import annotations

import concurrent.futures
import glob
import hashlib
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libigemm.so")
STAMP = LIB + ".sha256"
ARCH = "gfx950"

# Packed fp32 instructions are kept out of every HIP build of this library.
HIP_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) +
                  glob.glob(os.path.join(CSRC, "*.cpp")))


def headers():
    return sorted(glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(INCLUDE, "*.h")))


def compile_flags(extra_flags=None):
    base = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Wno-unused-parameter", "-I", INCLUDE, "-I", CSRC] + HIP_FLAGS
    return base + list(extra_flags or [])


def _hash_files(paths, flags) -> str:
    # Paths inside the repository enter relative to its root, so that the
    # same tree hashes the same wherever it is checked out.
    h = hashlib.sha256()
    h.update(" ".join(os.path.relpath(f, ROOT) if f.startswith(ROOT) else f
                      for f in flags).encode())
    for p in paths:
        h.update(os.path.relpath(p, ROOT).encode())
        with open(p, "rb") as f:
            h.update(hashlib.sha256(f.read()).digest())
    return h.hexdigest()


def source_hash(extra_flags=None) -> str:
    """SHA-256 over every source and header of the library and the flags."""
    return _hash_files(sources() + headers(), compile_flags(extra_flags))


# Everything the packed multiply kernel is built from (its source and the
# headers it includes); with the compile flags this names one build of it.
PACKED_KERNEL_SOURCES = [os.path.join(CSRC, f) for f in
                         ("igemm_packed.hip", "igemm_device.h", "igemm_internal.h")] + \
                        [os.path.join(INCLUDE, "igemm.h")]


def packed_kernel_hash() -> str:
    """SHA-256 of the packed kernel's sources and the compile flags: profile
    summaries taken on one build are reported only for the same build."""
    return _hash_files(PACKED_KERNEL_SOURCES, compile_flags())


# The same for the direct kernels (igemm_direct.hip and its headers).
DIRECT_KERNEL_SOURCES = [os.path.join(CSRC, f) for f in
                         ("igemm_direct.hip", "igemm_lds.h", "igemm_device.h",
                          "igemm_internal.h")] + [os.path.join(INCLUDE, "igemm.h")]


def direct_kernel_hash() -> str:
    return _hash_files(DIRECT_KERNEL_SOURCES, compile_flags())


def kernel_hash(family: str) -> str:
    """Hash of one kernel family's build: "packed" or "direct"."""
    return {"packed": packed_kernel_hash, "direct": direct_kernel_hash}[family]()


def is_current() -> bool:
    """True if the built library exists and was built from this tree."""
    try:
        with open(STAMP) as f:
            stamp = f.read().strip()
    except OSError:
        return False
    return os.path.exists(LIB) and stamp == source_hash()


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False, extra_flags=None, jobs: int = 0, object_cache=None) -> str:
    """Compile every source to an object (in parallel, ``jobs`` at a time;
    0 = one per CPU, at most 16) and link the shared library.

    object_cache: optional directory of objects keyed by the hash of their
    source, the headers and the flags; an object found there is reused
    instead of compiled (for quick rebuilds while editing one file). By
    default every source is compiled."""
    flags = compile_flags(extra_flags)
    base = [hipcc()] + flags
    srcs = sources()
    hdr_hash = _hash_files(headers(), flags)
    jobs = jobs or min(16, os.cpu_count() or 1)
    with tempfile.TemporaryDirectory(prefix="igemm_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in srcs]
        todo = []
        for s, o in zip(srcs, objs):
            if object_cache:
                key = _hash_files([s], [hdr_hash])
                cached = os.path.join(object_cache, f"{os.path.basename(s)}.{key[:20]}.o")
                if os.path.exists(cached):
                    shutil.copyfile(cached, o)
                    continue
                todo.append((s, o, cached))
            else:
                todo.append((s, o, None))
        with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as pool:
            futs = [pool.submit(_run, base + ["-c", s, "-o", o], verbose) for s, o, _ in todo]
            for f in futs:
                f.result()
        for s, o, cached in todo:
            if cached:
                os.makedirs(object_cache, exist_ok=True)
                shutil.copyfile(o, cached)
        tmp = LIB + ".tmp"
        _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", tmp],
             verbose)
    os.replace(tmp, LIB)
    with open(STAMP, "w") as f:
        f.write(source_hash(extra_flags) + "\n")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
