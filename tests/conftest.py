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
    build them when a fresh checkout has not been built yet.  So is the HIP
    library, when it is missing and hipcc is there (it cross-compiles for
    gfx950 without a GPU); a checkout that was built keeps its library."""
    import oracle
    from paper_2512_22147_amd import build as pkg_build
    from paper_2512_22147_amd import datagen

    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()
    if not os.path.exists(datagen.LIB_PATH):
        datagen.build()
    if not os.path.exists(pkg_build.LIB_PATH) and os.path.exists(pkg_build.HIPCC):
        pkg_build.build_mep()


_ensure_host_libs()


@pytest.fixture(scope="session")
def orc():
    import oracle

    return oracle.default()
