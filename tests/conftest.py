import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU oracle case")


def _ensure_built():
    lib = os.path.join(ROOT, "paper_2505_18629_amd", "librv.so")
    if not os.path.exists(lib):
        from __graft_entry__ import _build_script
        _build_script().build()
    orc = os.path.join(ROOT, "oracle", "liboracle_weights.so")
    if not os.path.exists(orc):
        import oracle
        oracle.build()


_ensure_built()


@pytest.fixture(scope="session")
def rv():
    import paper_2505_18629_amd as rv_mod
    return rv_mod


@pytest.fixture(scope="session")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    return torch.device("cuda:0")
