"""The CPU oracle against its pins (no GPU needed)."""
import numpy as np
import pytest

import oracle
import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle.igemm)


def test_golden_file_parses():
    cases = pins.load_golden()
    assert len(cases) >= 8
    assert {c["dtype"] for c in cases} == {"i16", "i8"}


def test_invalid_arguments_rejected():
    a = np.zeros(16, np.int16)
    c = np.zeros(16, np.int32)
    assert oracle.igemm_raw("i16", -1, 2, 2, a, 2, a, 2, c, 2) == -1
    assert oracle.igemm_raw("i16", 2, 2, 2, a, 1, a, 2, c, 2) == -1   # lda < k
    assert oracle.igemm_raw("i16", 2, 2, 2, a, 2, a, 1, c, 2) == -1   # ldb < n
    assert oracle.igemm_raw("i16", 2, 2, 2, a, 2, a, 2, c, 1) == -1   # ldc < n
    assert oracle.igemm_raw("i8", 0, 2, 2, a, 2, a, 2, c, 2) == 0     # no-op


def test_medium_random_against_numpy():
    """A larger shape with ragged sizes, still exact against numpy int64."""
    rng = np.random.default_rng(7)
    m, n, k = 301, 257, 515
    A = rng.integers(-32768, 32767, size=(m, k), dtype=np.int16, endpoint=True)
    B = rng.integers(-32768, 32767, size=(k, n), dtype=np.int16, endpoint=True)
    C0 = rng.integers(-(1 << 31), (1 << 31) - 1, size=(m, n), dtype=np.int32, endpoint=True)
    C = C0.copy()
    oracle.igemm(A, B, C)
    assert np.array_equal(C, pins.numpy_reference(A, B, C0))


def test_thread_count_does_not_change_result(tmp_path):
    """The OpenMP row split cannot change the result: 1 thread vs default."""
    import subprocess, sys, os
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import sys, numpy as np; sys.path.insert(0, %r); import oracle, workloads;"
        "A,B,C=workloads.random_operands('i16',97,131,263,seed=3);"
        "oracle.igemm(A,B,C); np.save(sys.argv[1], C)" % root)
    outs = []
    for nt in ("1", "5"):
        p = tmp_path / f"c{nt}.npy"
        env = dict(os.environ, OMP_NUM_THREADS=nt)
        subprocess.run([sys.executable, "-c", code, str(p)], check=True, env=env)
        outs.append(np.load(p))
    assert np.array_equal(outs[0], outs[1])
