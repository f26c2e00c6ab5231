import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP library)")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session", autouse=True)
def _built_cpu_libs():
    """The oracle and the input generator are plain C; build them if they are missing."""
    import gmm_synth
    import oracle
    gmm_synth.build_lib(force=False)
    oracle.build_lib(force=False)
