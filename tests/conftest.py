import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

_POOL = {}


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_collection_finish(session):
    # The oracle's worker processes are spawned here, after collection and
    # before any test initialises the GPU runtime, and only when a selected
    # test asks for them.
    if session.config.option.collectonly:
        return
    if any("oracle_pool" in getattr(item, "fixturenames", ()) for item in session.items):
        from oracle.parallel import OraclePool
        _POOL["pool"] = OraclePool()
        print(f"\n[oracle pool] {_POOL['pool'].workers} worker processes", flush=True)


def pytest_unconfigure(config):
    pool = _POOL.pop("pool", None)
    if pool is not None:
        pool.close()


@pytest.fixture(scope="session")
def oracle_pool():
    """Worker processes running the oracle on staged logits rows."""
    if "pool" not in _POOL:
        pytest.skip("oracle pool not started")
    return _POOL["pool"]


@pytest.fixture(scope="session")
def gpu():
    """The HIP binding, on a machine with a GPU (skips elsewhere)."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2606_02955_amd as fd
    fd.load()            # raises if the built library is missing
    return fd
