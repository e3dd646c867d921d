import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def layup_ctx():
    """A small context whose workspace holds the disagreement partial sums."""
    from paper_2410_05985_amd import layup as LU
    m = LU.Model(LU.mlp_config((8, 8), 4), "sgd")
    yield m.ctx
    m.close()
