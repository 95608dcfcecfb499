import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _ensure_host_libs():
    """The generator and the oracle are plain gcc builds of one C file each;
    build them when a fresh checkout has not been built yet."""
    import oracle
    from paper_2512_22147_amd import datagen

    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()
    if not os.path.exists(datagen.LIB_PATH):
        datagen.build()


_ensure_host_libs()


@pytest.fixture(scope="session")
def orc():
    import oracle

    return oracle.default()
