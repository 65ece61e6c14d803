import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

_LIBS = (
    os.path.join(ROOT, "oracle", "liboracle.so"),
    os.path.join(ROOT, "workloads", "libgen.so"),
    os.path.join(ROOT, "paper_2609_18178_amd", "libpactshard.so"),
    os.path.join(ROOT, "tests", "native", "c_caller"),
)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds")
    # Build only when nothing is built; a present library is used as is.
    missing = [os.path.relpath(p, ROOT) for p in _LIBS if not os.path.exists(p)]
    if missing:
        subprocess.run(["make", "-C", ROOT, "-j8"] + missing, check=True)


@pytest.fixture(scope="session")
def root():
    return ROOT
