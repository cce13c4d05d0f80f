import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU oracle test")


def read_fixture(name):
    """Non-comment, non-empty lines of tests/golden/<name>, split on whitespace."""
    path = os.path.join(ROOT, "tests", "golden", name)
    with open(path) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.lstrip().startswith("#")]


@pytest.fixture(scope="session")
def built_lib():
    """Path of libmdlstm.so; built in-tree only if nothing is built yet."""
    from paper_1902_11208_amd import _lib

    if not os.path.exists(_lib.LIB_PATH):
        from paper_1902_11208_amd import build

        build.build()
    return _lib.LIB_PATH


def rel_err(got, ref):
    """Normwise L2 relative error ||got - ref||_2 / ||ref||_2 (the parity metric)."""
    import numpy as np

    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.linalg.norm(ref.ravel())) if ref.size else 0.0
    num = float(np.linalg.norm((got - ref).ravel())) if ref.size else 0.0
    return num / den if den > 0 else num


def rel_max(got, ref):
    """max|got - ref| / max|ref| (reported, and bounded by a looser guard)."""
    import numpy as np

    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    return num / den if den > 0 else num
