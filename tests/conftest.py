import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def oracle_lib():
    from oracle.oracle import load_oracle
    return load_oracle()


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library, loaded after torch; fails (does not skip) if missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible to torch")
    import paper_2608_01563_amd as mg
    mg.load_library()
    return mg
