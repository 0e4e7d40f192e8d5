import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads")


def _gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def gpu():
    """The HIP path on cuda:0; skips on a machine without a GPU.

    On a machine with a GPU the library must load: a missing build is an error,
    never a silent fallback.
    """
    if not _gpu_available():
        pytest.skip("no GPU on this machine")
    import paper_2608_17995_amd as avits
    avits.load()  # raises if libavits.so is missing
    return avits


def pytest_sessionstart(session):
    # A child run of the oracle pins with one planted mistake (see
    # tests/oracle_mistakes.py); never set in an ordinary run.
    name = os.environ.get("AVITS_PLANT_MISTAKE")
    if name:
        sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
        import oracle_mistakes
        oracle_mistakes.plant(name)
