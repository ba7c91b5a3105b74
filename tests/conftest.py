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
    """Build the HIP library and the oracle when they are missing or were
    built from other sources than the tree's (each build stamps the SHA-256 of
    its sources, headers and flags next to the library)."""
    from paper_2302_07594_amd import build as hip_build
    from oracle import build as oracle_build
    if not hip_build.is_current():
        hip_build.build()
    if not oracle_build.is_current():
        oracle_build.build()


_ensure_built()
