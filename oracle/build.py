"""Build the CPU oracle library (test infrastructure) with the host C compiler.

``python oracle/build.py`` or ``oracle.build.build()`` writes
``oracle/liboracle.so``, and ``liboracle.so.sha256`` beside it with the
SHA-256 of the source and the compiler command (``is_current()`` compares
it with the tree). ``build_sanitized()`` writes a separate copy built with
the address and undefined-behaviour sanitizers for the sanitizer test. The
GPU library is built separately and shares no source with this one.
"""
from __future__ import annotations

import hashlib
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "igemm_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
STAMP = LIB + ".sha256"
SAN_LIB = os.path.join(HERE, "liboracle_san.so")

FLAGS = ["-std=c11", "-O3", "-march=x86-64-v3", "-fopenmp", "-fPIC", "-shared", "-Wall",
         "-Wextra", "-Werror"]
SAN_FLAGS = ["-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-fPIC",
             "-shared", "-Wall", "-Wextra", "-Werror", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all"]


def _cc():
    return os.environ.get("CC", "gcc")


def source_hash() -> str:
    h = hashlib.sha256()
    h.update(" ".join([_cc()] + FLAGS).encode())
    with open(SRC, "rb") as f:
        h.update(f.read())
    return h.hexdigest()


def is_current() -> bool:
    try:
        with open(STAMP) as f:
            return os.path.exists(LIB) and f.read().strip() == source_hash()
    except OSError:
        return False


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [_cc()] + FLAGS + [SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    with open(STAMP, "w") as f:
        f.write(source_hash() + "\n")
    return LIB


def build_sanitized(out: str = SAN_LIB) -> str:
    """The oracle built with -fsanitize=address,undefined (any report aborts);
    load it into a process that preloads the sanitizer runtime."""
    tmp = out + ".tmp"
    subprocess.run([_cc()] + SAN_FLAGS + [SRC, "-o", tmp], check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
