import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size cases (minutes of CPU work)")


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


@pytest.fixture(scope="session")
def lib():
    """The HIP library on a real GPU. Fails (does not skip) when the library is missing."""
    import torch

    import paper_2608_20530_amd as L

    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    L.load_library()
    return L


_CFG_CACHE = {}


@pytest.fixture(scope="session")
def cfg_inputs():
    """cfg_inputs(i) -> (cfg, dict of CPU tensors), generated once per session."""
    import workloads

    def get(i):
        if i not in _CFG_CACHE:
            cfg = workloads.config(i)
            _CFG_CACHE[i] = (cfg, workloads.make_inputs(cfg))
        return _CFG_CACHE[i]

    return get
