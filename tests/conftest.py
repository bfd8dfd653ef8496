import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU oracle case")
    config.addinivalue_line("markers", "sanitize: the CPU suite rebuilt and rerun under "
                            "AddressSanitizer and UndefinedBehaviorSanitizer")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle
