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


_CHAIN_CACHE = {}


@pytest.fixture(scope="session")
def oracle_chain(cfg_inputs):
    """oracle_chain(i) -> the oracle chain of every request of workload i (parity.oracle_chain_all),
    computed once per session on a thread pool."""
    import time

    from parity import oracle_chain_all, oracle_threads

    def get(i):
        if i not in _CHAIN_CACHE:
            cfg, inp = cfg_inputs(i)
            t0 = time.perf_counter()
            _CHAIN_CACHE[i] = oracle_chain_all(cfg, inp)
            print(f"oracle chain of config {i} ({cfg.N} requests) in "
                  f"{time.perf_counter() - t0:.1f} s on {oracle_threads()} threads", flush=True)
        return _CHAIN_CACHE[i]

    return get
