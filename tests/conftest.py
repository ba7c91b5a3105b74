import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds")


def _ensure_built():
    """Build the HIP library and the oracle only if nothing is built yet."""
    lib = os.path.join(ROOT, "paper_2302_07594_amd", "libigemm.so")
    if not os.path.exists(lib):
        from paper_2302_07594_amd import build as hip_build
        hip_build.build()
    olib = os.path.join(ROOT, "oracle", "liboracle.so")
    if not os.path.exists(olib):
        from oracle import build as oracle_build
        oracle_build.build()


_ensure_built()
